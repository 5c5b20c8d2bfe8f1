"""Input generators: determinism and the structural properties the workloads
promise (CPU only)."""
import numpy as np
import torch

import synth


def test_feistel_is_a_permutation():
    for n in (1, 2, 3, 10, 1000, 4097, 100_003):
        x = torch.arange(n, dtype=torch.int64)
        y = synth.feistel_permute(x, n, 12345)
        assert torch.equal(torch.sort(y).values, x)


def test_uniform_graph_properties():
    off, idx = synth.uniform_graph(2000, 1, 20, 0)
    deg = np.diff(off)
    assert deg.min() >= 1 and deg.max() <= 20
    assert abs(deg.mean() - 10.5) < 0.5
    for v in range(0, 2000, 37):
        row = idx[off[v]:off[v + 1]]
        assert np.all(np.diff(row) > 0) and v not in row and row.min() >= 0 and row.max() < 2000
    off2, idx2 = synth.uniform_graph(2000, 1, 20, 0)
    assert np.array_equal(off, off2) and np.array_equal(idx, idx2)


def test_rmat_graph_properties():
    n = 5000
    off, idx = synth.rmat_graph(n, 60_000, 0.57, 0.19, 0.19, 0)
    assert off[0] == 0 and int(off[-1]) == idx.numel() and off.numel() == n + 1
    assert bool((off[1:] >= off[:-1]).all())
    src = torch.repeat_interleave(torch.arange(n), off[1:] - off[:-1])
    key = src * n + idx.long()
    assert bool((key[1:] > key[:-1]).all())          # rows sorted, no duplicates
    assert not bool((src == idx.long()).any())       # no self loops
    assert idx.min() >= 0 and idx.max() < n
    deg = (off[1:] - off[:-1]).float()
    assert deg.max() > 10 * deg.mean()               # heavy tail
    off2, idx2 = synth.rmat_graph(n, 60_000, 0.57, 0.19, 0.19, 0)
    assert torch.equal(off, off2) and torch.equal(idx, idx2)
    # chunking does not change the draws
    k1 = synth.rmat_edges(n, 60_000, 0.57, 0.19, 0.19, 0, chunk=7_000)
    assert torch.equal(k1, key)


def test_seeds_and_cache():
    s = synth.seed_batches(10_000, 4, 64, 0)
    assert s.shape == (4, 64) and s.unique().numel() == 256
    assert s.min() >= 0 and s.max() < 10_000
    idx = torch.tensor([3, 3, 3, 1, 1, 2, 0, 4, 4, 4], dtype=torch.int32)
    slot, nodes = synth.cache_by_indegree(idx, 6, 3)
    assert nodes.tolist() == [3, 4, 1]               # in-degree 3, 3, 2: ties by ID
    assert slot.tolist() == [-1, 2, -1, 0, 1, -1]


def test_tiny_workload_is_deterministic():
    a = synth.make_workload("T")
    b = synth.make_workload("T")
    assert torch.equal(a.offsets, b.offsets) and torch.equal(a.indices, b.indices)
    assert torch.equal(a.seeds, b.seeds) and torch.equal(a.feats, b.feats)
    assert a.cache.shape == (1000, 16)
    assert torch.equal(a.cache, a.feats[a.cache_nodes])


def test_seeds_skip_isolated_nodes():
    n = 3000
    off, idx = synth.rmat_graph(n, 20_000, 0.57, 0.19, 0.19, 0)
    deg = off[1:] - off[:-1]
    assert int((deg == 0).sum()) > 0
    s = synth.seed_batches(n, 4, 100, 0, offsets=off)
    assert s.unique().numel() == 400
    assert bool((deg[s.long()] > 0).all())
    # with every node eligible the walk is the plain keyed permutation
    full = torch.ones(n + 1, dtype=torch.int64).cumsum(0) - 1
    assert torch.equal(synth.seed_batches(n, 4, 100, 0, offsets=full),
                       synth.seed_batches(n, 4, 100, 0))
