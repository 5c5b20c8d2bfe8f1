"""Loops over groups with the mask-clearing flags: sampling with
DG_SAMPLE_EXIT_CLEAR (and DG_SAMPLE_ENTRY_CLEAR from the second group on),
packing with DG_PACK_CLEAR_MEMBERSHIP and the member-lines map sampling
writes, on one workspace per call and one membership buffer.  Every output must equal that of independent calls without
the flags, the membership output must equal theirs, and packing must leave the
mask all-zero.  The workspaces and the mask start filled with garbage, which
the first call (without DG_SAMPLE_ENTRY_CLEAR) must not see."""
import random

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def dg():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2405_05231_amd as m
    return m


def same_sample(a, b):
    assert np.array_equal(a.hop_ptr, b.hop_ptr) and np.array_equal(a.edge_ptr, b.edge_ptr)
    for bb in range(a.hop_ptr.shape[0]):
        n, e = int(a.hop_ptr[bb, -1]), int(a.edge_ptr[bb, -1])
        assert torch.equal(a.nodes[bb, :n], b.nodes[bb, :n]), bb
        assert torch.equal(a.edge_src[bb, :e], b.edge_src[bb, :e]), bb
        assert torch.equal(a.edge_dst[bb, :e], b.edge_dst[bb, :e]), bb


def same_pack(a, b, counts, keys=None):
    """keys: the size fields to compare (default all of them)."""
    if keys is None:
        assert a.sizes == b.sizes
    else:
        assert {k: a.sizes[k] for k in keys} == {k: b.sizes[k] for k in keys}
    rows = a.sizes["packed_rows"]
    assert np.array_equal(a.packed_ptr_host, b.packed_ptr_host)
    assert torch.equal(a.packed_ids[:rows], b.packed_ids[:rows])
    assert torch.equal(a.packed[:rows], b.packed[:rows])
    nu = a.sizes["unique_nodes"]
    assert torch.equal(a.unique[:nu], b.unique[:nu])
    for bb, n in enumerate(counts):
        assert torch.equal(a.loc[bb, :int(n)], b.loc[bb, :int(n)]), bb


def sparse_graph(fan=(3, 3, 2)):
    """200k nodes, degrees 0..6, 4 batches of 16 seeds: every hop is small
    enough to use touched marks, except that the last one reads every word when
    the call asks for the member-lines map or a clear exit.  With a last
    fan-out of 0 the last hop runs no count pass, and the sampler writes the map
    with a pass of its own and clears its state with a fill."""
    n = 200_000
    off, idx = synth.uniform_graph(n, 0, 6, seed=31)
    rnd = random.Random(99)
    gen = torch.Generator().manual_seed(3)
    feats = torch.randn((n, 4), generator=gen).to(DEV)
    slot = torch.full((n,), -1, dtype=torch.int32)
    slot[torch.tensor(rnd.sample(range(n), n // 10))] = torch.arange(n // 10, dtype=torch.int32)
    seeds = [torch.tensor([rnd.sample(range(n), 16) for _ in range(4)], dtype=torch.int32,
                          device=DEV) for _ in range(3)]
    return (torch.from_numpy(off).to(DEV), torch.from_numpy(idx).to(DEV), feats, slot.to(DEV),
            seeds, list(fan), 1234)


def workload_groups(name):
    w = synth.make_workload(name, device=DEV)
    cfg = w.cfg
    seeds = [synth.seed_batches(cfg.n, cfg.B, cfg.S, cfg.seed + 1 + g, DEV, offsets=w.offsets)
             for g in range(3)]
    return w.offsets, w.indices, w.feats, w.cache_slot, seeds, list(cfg.fanouts), w.rng_seed


def case_inputs(case):
    if case == "sparse":
        return sparse_graph()
    if case == "sparse_f0":
        return sparse_graph((3, 3, 0))
    return workload_groups(case)


@pytest.mark.parametrize("case,layered,direct", [("M1", False, True), ("M1", False, False),
                                                 ("M1", True, True), ("sparse", False, True),
                                                 ("sparse_f0", False, True)])
def test_group_loop_with_clear_flags(dg, case, layered, direct):
    off, idx, feats, slot, groups, fan, rng = case_inputs(case)
    N = off.numel() - 1
    B, S = groups[0].shape
    node_cap, edge_cap = dg.sample_bounds(N, idx.numel(), S, fan, layered)
    flags = dg.sample_flags(layered, direct)
    ws_s = torch.full((dg._L.dg_sample_workspace_bytes(N, B, node_cap, edge_cap, flags),), 0xA5,
                      dtype=torch.uint8, device=DEV)
    mem = torch.full((N,), -1, dtype=torch.int64, device=DEV)
    lines = torch.full((dg.member_lines_bytes(N),), 0xAB, dtype=torch.uint8, device=DEV)
    ws_p = None
    for g, seeds in enumerate(groups):
        print(f"[{case} layered={layered} direct={direct}] group {g}", flush=True)
        sr = dg.sample_group(off, idx, seeds, fan, rng, batch_base=g * B, membership=mem,
                             workspace=ws_s, layered=layered, direct=direct, exit_clear=True,
                             entry_clear=g > 0, member_lines=lines)
        mem_f = torch.empty(N, dtype=torch.int64, device=DEV)
        sr_f = dg.sample_group(off, idx, seeds, fan, rng, batch_base=g * B, membership=mem_f,
                               layered=layered, direct=direct)
        same_sample(sr, sr_f)
        assert torch.equal(mem, mem_f)
        counts = sr.hop_ptr[:, -1].copy()
        if ws_p is None:
            ws_p = torch.full((dg._L.dg_pack_workspace_bytes(N, B, int(counts.sum())) * 2,), 0x5A,
                              dtype=torch.uint8, device=DEV)
        pr = dg.pack_group(feats, slot, sr.nodes, counts, with_unique=True, membership=mem,
                           workspace=ws_p, clear_membership=True, member_lines=lines)
        torch.cuda.synchronize()
        assert int(mem.count_nonzero()) == 0
        pr_f = dg.pack_group(feats, slot, sr_f.nodes, counts, with_unique=True, membership=mem_f)
        same_pack(pr, pr_f, counts)


def lines_ref(dg, mem):
    """The member-lines map computed from the membership words by torch."""
    N = mem.numel()
    nbytes = dg.member_lines_bytes(N)
    pad = torch.zeros(nbytes * 8, dtype=torch.int64, device=DEV)
    pad[:N] = mem
    return (pad.view(-1, 8) != 0).any(dim=1)


@pytest.mark.parametrize("case,layered,direct", [("M1", False, True), ("M1", True, False),
                                                 ("sparse", False, True),
                                                 ("sparse_f0", False, True)])
def test_member_lines(dg, case, layered, direct):
    """The map sampling writes (by its last count pass, or by a pass of its own
    when the last hop runs none) marks exactly the 8-node lines that hold a
    member; packing with it gives the outputs of packing without it, and a map
    that misses a member line is reported."""
    off, idx, feats, slot, groups, fan, rng = case_inputs(case)
    N = off.numel() - 1
    seeds = groups[0]
    B = seeds.shape[0]
    mem = torch.empty(N, dtype=torch.int64, device=DEV)
    lines = torch.full((dg.member_lines_bytes(N),), 0xAB, dtype=torch.uint8, device=DEV)
    sr = dg.sample_group(off, idx, seeds, fan, rng, membership=mem, member_lines=lines,
                         layered=layered, direct=direct)
    torch.cuda.synchronize()
    assert torch.equal(lines != 0, lines_ref(dg, mem))
    counts = sr.node_count
    ref = dg.pack_group(feats, slot, sr.nodes, counts, with_unique=True, membership=mem)
    mem2 = mem.clone()
    got = dg.pack_group(feats, slot, sr.nodes, counts, with_unique=True, membership=mem2,
                        member_lines=lines, clear_membership=True)
    torch.cuda.synchronize()
    assert int(mem2.count_nonzero()) == 0
    same_pack(got, ref, counts)
    # a map that misses a line holding a member
    bad = lines.clone()
    bad[int((lines != 0).nonzero()[0])] = 0
    with pytest.raises(dg.DGError) as e:
        dg.pack_group(feats, slot, sr.nodes, counts, membership=mem, member_lines=bad)
    assert e.value.status == -1
