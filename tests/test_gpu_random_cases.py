"""Seeded random sweeps of valid configurations.

1. Small configurations, bit-exact against the CPU oracle through the whole
   path (sample -> pack -> assemble): graph size and degree range, batch count
   (1 to 64, around the 32-bit and 64-bit word sizes), seeds per batch, hop
   count, fan-outs (0, all neighbours, below / at / above the register path),
   row sizes from 1 byte to 4 KiB in several dtypes, cache shares from none to
   every node, both frontier rules and both relabelling modes.
2. Loops of three groups on one workspace and one membership buffer with the
   clearing flags and the member-lines map, on graphs of up to 300k nodes (so
   that hops fall on both sides of the touched-marks limit): every group's
   outputs must equal those of independent calls without the flags, and
   packing must leave the mask all-zero.
3. Both of the above through the one-call path (dg_sample_pack_group).
4. Frequency-ranked cache selection and the MinHash disk-cache order on random
   small groups, bit-exact against the oracle.

Each case is fixed by its index, so a failure names a reproducible
configuration."""
import random

import numpy as np
import pytest
import torch

from test_gpu_clear import same_pack, same_sample
from test_gpu_parity import check_all, random_case

pytestmark = pytest.mark.gpu
DEV = "cuda"

N_CASES = 200
N_LOOP_CASES = 16

ROW_SHAPES = [(1, torch.uint8), (3, torch.uint8), (7, torch.int16), (4, torch.float32),
              (16, torch.float32), (8, torch.float16), (24, torch.float16),
              (128, torch.float32), (384, torch.float16), (385, torch.float32),
              (768, torch.float16), (1024, torch.float32)]
FANOUTS = [-1, 0, 1, 2, 3, 5, 8, 15, 16, 17, 25, 33, 40]


def make_case(i):
    rnd = random.Random(7000 + i)
    n = rnd.choice([1, 2, 3, 17, 64, 100, 257, 1000, 3000])
    big = n >= 1000
    maxdeg = rnd.randint(0, min(n - 1, 20 if big else 80)) if n > 1 else 0
    B = rnd.choice([1, 2, 5, 16] if big else [1, 2, 5, 31, 32, 33, 63, 64])
    S = rnd.randint(1, min(n, 40))
    K = rnd.randint(1, 3 if big else 4)
    fan = [rnd.choice(FANOUTS) for _ in range(K)]
    dim, dtype = rnd.choice(ROW_SHAPES)
    share = rnd.choice([0.0, 0.01, 0.1, 0.5, 1.0])
    layered = rnd.random() < 0.3
    direct = rnd.random() < 0.5
    return rnd, dict(n=n, maxdeg=maxdeg, B=B, S=S, fan=fan, dim=dim, dtype=dtype, share=share,
                     layered=layered, direct=direct)


@pytest.fixture(scope="module")
def dg():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2405_05231_amd as m
    return m


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_valid_case(dg, orc, case):
    rnd, c = make_case(case)
    print(f"case {case}: {c}", flush=True)
    n = c["n"]
    if c["maxdeg"]:
        off, idx = random_case(rnd, n, c["maxdeg"])
    else:
        off, idx = torch.zeros(n + 1, dtype=torch.int64), torch.zeros(0, dtype=torch.int32)
    seeds = torch.tensor([rnd.sample(range(n), c["S"]) for _ in range(c["B"])], dtype=torch.int32)
    gen = torch.Generator().manual_seed(case)
    if c["dtype"].is_floating_point:
        feats = torch.randn((n, c["dim"]), generator=gen).to(c["dtype"])
    else:
        feats = torch.randint(0, 100, (n, c["dim"]), generator=gen).to(c["dtype"])
    ncache = int(n * c["share"])
    cache_nodes = torch.tensor(rnd.sample(range(n), ncache), dtype=torch.int64)
    slot = torch.full((n,), -1, dtype=torch.int32)
    slot[cache_nodes] = torch.arange(ncache, dtype=torch.int32)
    check_all(dg, orc, off, idx, seeds, c["fan"], 4242 + case, feats, slot, cache_nodes,
              batch_base=3 * case, sample_kw={"layered": c["layered"], "direct": c["direct"]})
    if c["direct"]:
        # the same case in one dg_sample_pack_group call: with the direct table
        # the last hop's compaction also does packing's pass
        check_all(dg, orc, off, idx, seeds, c["fan"], 4242 + case, feats, slot, cache_nodes,
                  batch_base=3 * case,
                  sample_kw={"layered": c["layered"], "direct": True, "handoff": "fused"})


def strided_graph(nrng, n, dmax):
    """Each node v gets U{0..dmax} distinct out-neighbours v + step_v * k (mod n),
    k = 1..d, with step_v * dmax < n (so none is v itself); rows sorted."""
    deg = nrng.integers(0, dmax + 1, n)
    step = nrng.integers(1, max(2, n // (dmax + 1)), n)
    k = np.arange(1, dmax + 1)
    nb = (np.arange(n)[:, None] + step[:, None] * k[None, :]) % n
    nb = np.sort(np.where(k[None, :] <= deg[:, None], nb, n), axis=1)
    idx = nb[np.arange(dmax)[None, :] < deg[:, None]].astype(np.int32)
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(deg)
    return torch.from_numpy(off), torch.from_numpy(idx)


def make_loop_case(i):
    rnd = random.Random(9100 + i)
    c = dict(n=rnd.choice([5000, 60000, 300000]), dmax=rnd.choice([2, 6, 20]),
             B=rnd.choice([1, 7, 32, 64]), S=rnd.choice([1, 4, 16]), K=rnd.randint(1, 3),
             layered=rnd.random() < 0.3, direct=rnd.random() < 0.5,
             dim=rnd.choice([4, 16, 128]), share=rnd.choice([0.0, 0.05, 0.5]))
    choices = [1, 3, 5, 10, 25] if c["layered"] else [-1, 1, 3, 5, 10, 25]
    c["fan"] = [rnd.choice(choices) for _ in range(c["K"])]
    return rnd, c


@pytest.mark.parametrize("case", range(N_LOOP_CASES))
def test_random_group_loop_with_flags(dg, case):
    rnd, c = make_loop_case(case)
    print(f"loop case {case}: {c}", flush=True)
    n, B, S = c["n"], c["B"], c["S"]
    nrng = np.random.default_rng(case)
    off_h, idx_h = strided_graph(nrng, n, c["dmax"])
    off, idx = off_h.to(DEV), idx_h.to(DEV)
    gen = torch.Generator().manual_seed(case)
    feats = torch.randn((n, c["dim"]), generator=gen).to(DEV)
    ncache = int(n * c["share"])
    slot = torch.full((n,), -1, dtype=torch.int32)
    slot[torch.tensor(rnd.sample(range(n), ncache), dtype=torch.int64)] = \
        torch.arange(ncache, dtype=torch.int32)
    slot = slot.to(DEV)
    groups = [torch.tensor([rnd.sample(range(n), S) for _ in range(B)], dtype=torch.int32,
                           device=DEV) for _ in range(3)]
    fan, rng, layered, direct = c["fan"], 777 + case, c["layered"], c["direct"]
    node_cap, edge_cap = dg.sample_bounds(n, idx.numel(), S, fan, layered)
    flags = dg.sample_flags(layered, direct)
    ws_s = torch.full((dg._L.dg_sample_workspace_bytes(n, B, node_cap, edge_cap, flags),), 0xA5,
                      dtype=torch.uint8, device=DEV)
    mem = torch.full((n,), -1, dtype=torch.int64, device=DEV)
    lines = torch.full((dg.member_lines_bytes(n),), 0xAB, dtype=torch.uint8, device=DEV)
    ws_p = None
    for g, seeds in enumerate(groups):
        sr = dg.sample_group(off, idx, seeds, fan, rng, batch_base=g * B, membership=mem,
                             workspace=ws_s, layered=layered, direct=direct, exit_clear=True,
                             entry_clear=g > 0, member_lines=lines)
        mem_f = torch.empty(n, dtype=torch.int64, device=DEV)
        sr_f = dg.sample_group(off, idx, seeds, fan, rng, batch_base=g * B, membership=mem_f,
                               layered=layered, direct=direct)
        same_sample(sr, sr_f)
        assert torch.equal(mem, mem_f), g
        counts = sr.hop_ptr[:, -1].copy()
        need = dg._L.dg_pack_workspace_bytes(n, B, int(counts.sum()))
        if ws_p is None or ws_p.numel() < need:
            ws_p = torch.full((need * 2,), 0x5A, dtype=torch.uint8, device=DEV)
        pr = dg.pack_group(feats, slot, sr.nodes, counts, with_unique=True, membership=mem,
                           workspace=ws_p, clear_membership=True, member_lines=lines)
        torch.cuda.synchronize()
        assert int(mem.count_nonzero()) == 0, g
        pr_f = dg.pack_group(feats, slot, sr_f.nodes, counts, with_unique=True, membership=mem_f)
        same_pack(pr, pr_f, counts)


@pytest.mark.parametrize("case", range(N_LOOP_CASES))
def test_random_group_loop_in_one_call(dg, case):
    """Three groups through dg_sample_pack_group on one sampling workspace, one
    packing workspace and one membership buffer (garbage in both workspaces at
    the start), clearing flags on: each group's outputs equal those of
    sample_group + pack_group on fresh buffers, and the membership words end
    all-zero.  One case in four relabels by hash, where packing's own passes
    follow sampling inside the call."""
    rnd, c = make_loop_case(case)
    direct = case % 4 != 3
    print(f"one-call loop case {case}: {c} direct={direct}", flush=True)
    n, B, S = c["n"], c["B"], c["S"]
    nrng = np.random.default_rng(500 + case)
    off_h, idx_h = strided_graph(nrng, n, c["dmax"])
    off, idx = off_h.to(DEV), idx_h.to(DEV)
    gen = torch.Generator().manual_seed(500 + case)
    feats = torch.randn((n, c["dim"]), generator=gen).to(DEV)
    ncache = int(n * c["share"])
    slot = torch.full((n,), -1, dtype=torch.int32)
    slot[torch.tensor(rnd.sample(range(n), ncache), dtype=torch.int64)] = \
        torch.arange(ncache, dtype=torch.int32)
    slot = slot.to(DEV)
    groups = [torch.tensor([rnd.sample(range(n), S) for _ in range(B)], dtype=torch.int32,
                           device=DEV) for _ in range(3)]
    fan, rng, layered = c["fan"], 991 + case, c["layered"]
    node_cap, edge_cap = dg.sample_bounds(n, idx.numel(), S, fan, layered)
    flags = dg.sample_flags(layered, direct, True, True)
    ws_s = torch.full((dg._L.dg_sample_workspace_bytes(n, B, node_cap, edge_cap, flags),), 0xA5,
                      dtype=torch.uint8, device=DEV)
    ws_p = torch.full((dg._L.dg_sample_pack_workspace_bytes(n, B, node_cap),), 0x5A,
                      dtype=torch.uint8, device=DEV)
    mem = torch.full((n,), -1, dtype=torch.int64, device=DEV)
    for g, seeds in enumerate(groups):
        sr, pr = dg.sample_pack_group(off, idx, seeds, fan, rng, feats, slot, batch_base=g * B,
                                      node_cap=node_cap, edge_cap=edge_cap, with_unique=True,
                                      workspace=ws_s, pack_workspace=ws_p, membership=mem,
                                      layered=layered, direct=direct, entry_clear=g > 0,
                                      exit_clear=True)
        torch.cuda.synchronize()
        assert int(mem.count_nonzero()) == 0, g
        sr_f = dg.sample_group(off, idx, seeds, fan, rng, batch_base=g * B, layered=layered,
                               direct=direct, node_cap=node_cap, edge_cap=edge_cap)
        same_sample(sr, sr_f)
        counts = sr_f.hop_ptr[:, -1].copy()
        pr_f = dg.pack_group(feats, slot, sr_f.nodes, counts, with_unique=True)
        # the one call also reports sampling's sizes; compare packing's
        same_pack(pr, pr_f, counts, keys=("packed_rows", "unique_nodes", "unique_packed"))
        assert pr.sizes["total_nodes"] == int(counts.sum()), g


N_NEXT_CASES = 30


def small_sampled(dg, case):
    """A random small graph and group, sampled on the device with the
    membership words kept; returns (n, B, mem, the batches' node lists, rnd)."""
    rnd = random.Random(12000 + case)
    n = rnd.choice([3, 40, 300, 2000])
    maxdeg = rnd.randint(0, min(n - 1, 30))
    B = rnd.choice([1, 3, 32, 33, 64])
    S = rnd.randint(1, min(n, 20))
    fan = [rnd.choice([-1, 1, 3, 8, 20]) for _ in range(rnd.randint(1, 3))]
    off, idx = (random_case(rnd, n, maxdeg) if maxdeg else
                (torch.zeros(n + 1, dtype=torch.int64), torch.zeros(0, dtype=torch.int32)))
    seeds = torch.tensor([rnd.sample(range(n), S) for _ in range(B)], dtype=torch.int32)
    mem = torch.empty(n, dtype=torch.int64, device=DEV)
    sr = dg.sample_group(off.to(DEV), idx.to(DEV), seeds.to(DEV), fan, 55 + case,
                         membership=mem, layered=rnd.random() < 0.3)
    lists = [sr.batch_nodes(b).cpu().numpy() for b in range(B)]
    return n, B, mem, lists, rnd


@pytest.mark.parametrize("case", range(N_NEXT_CASES))
def test_random_cache_by_frequency(dg, orc, case):
    n, B, mem, lists, rnd = small_sampled(dg, case)
    for C in sorted({0, 1, rnd.randint(0, n), n // 2, n}):
        print(f"cache case {case}: n={n} B={B} C={C}", flush=True)
        slot, nodes, cached = dg.cache_by_frequency(mem, B, C)
        r_slot, r_nodes, r_cached = orc.cache_by_frequency(n, lists, C)
        assert cached == r_cached, C
        assert np.array_equal(slot.cpu().numpy(), r_slot), C
        assert np.array_equal(nodes.cpu().numpy(), r_nodes), C


@pytest.mark.parametrize("case", range(N_NEXT_CASES))
def test_random_minhash_order(dg, orc, case):
    n, B, mem, lists, rnd = small_sampled(dg, case)
    k = rnd.choice([1, 2, 5])
    # disk-cache entries: a random subset of all nodes, accessed or not, in random order
    m = rnd.randint(1, n)
    entries = torch.tensor(rnd.sample(range(n), m), dtype=torch.int32, device=DEV)
    g = torch.Generator().manual_seed(case)
    perms = torch.stack([torch.randperm(B, generator=g) for _ in range(k)]).to(torch.int32)
    print(f"minhash case {case}: n={n} B={B} k={k} m={m}", flush=True)
    order, sig = dg.minhash_order(mem, B, entries, perms.to(DEV))
    r_order, r_sig = orc.minhash_order(n, lists, entries.cpu().numpy(), perms.numpy())
    assert np.array_equal(sig.cpu().numpy(), r_sig)
    assert np.array_equal(order.cpu().numpy(), r_order)
