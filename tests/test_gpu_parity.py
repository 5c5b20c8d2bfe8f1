"""Parity of the HIP path (through the C ABI) with the CPU oracle, bit-exact:
every output is an integer or a row copy, so the tolerance is zero.  Small
workloads compare every output element; edge cases cover empty and ragged
inputs, fan-outs below / at / above the degree, all-neighbour hops, fan-outs
beyond the register path, every cache share, odd row sizes and the group
split."""
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


def to_np(t):
    return t.detach().cpu().numpy()


def run_path(dg, off, idx, seeds, fanouts, rng_seed, feats, cache_slot, cache_nodes,
             batch_base=0, sample_kw=None):
    """The device path: sample -> pack -> assemble every batch.  With
    sample_kw["handoff"], sampling also writes the cached nodes' address-table
    entries (garbage in the table beforehand) and packing completes the rest
    (DG_PACK_LOC_PENDING)."""
    kw = dict(sample_kw or {})
    handoff = kw.pop("handoff", False)
    off_d, idx_d = off.to(DEV), idx.to(DEV)
    seeds_d = seeds.to(DEV)
    X = feats.to(DEV)
    slot = cache_slot.to(DEV)
    cache = X.index_select(0, cache_nodes.to(DEV)) if cache_nodes.numel() else None
    R = X[0].numel() * X.element_size()
    if handoff == "fused":
        # one dg_sample_pack_group call; garbage in every output beforehand
        B = seeds.shape[0]
        ncap, ecap = dg.sample_bounds(off.numel() - 1, idx.numel(), seeds.shape[1], fanouts,
                                      kw.get("layered", False))
        cap = B * ncap
        out = dg.PackResult(packed=torch.full((cap, R), 7, dtype=torch.uint8, device=DEV),
                            packed_ids=torch.full((cap,), -5, dtype=torch.int32, device=DEV),
                            packed_ptr=torch.full((B + 1,), -5, dtype=torch.int64, device=DEV),
                            packed_ptr_host=np.zeros(B + 1, dtype=np.int64),
                            loc=torch.full((B, ncap), -3, dtype=torch.int32, device=DEV),
                            unique=torch.full((cap,), -5, dtype=torch.int32, device=DEV),
                            sizes={}, timing=None, row_bytes=R)
        mem = torch.full((off.numel() - 1,), -1, dtype=torch.int64, device=DEV)
        sr, pr = dg.sample_pack_group(off_d, idx_d, seeds_d, fanouts, rng_seed, X, slot,
                                      batch_base=batch_base, node_cap=ncap, edge_cap=ecap,
                                      pack_out=out, membership=mem, exit_clear=True, **kw)
        assert int(torch.count_nonzero(mem)) == 0  # packing consumed the membership words
    elif not handoff:
        sr = dg.sample_group(off_d, idx_d, seeds_d, fanouts, rng_seed, batch_base=batch_base,
                             **kw)
        pr = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True)
    else:
        B = seeds.shape[0]
        ncap, ecap = dg.sample_bounds(off.numel() - 1, idx.numel(), seeds.shape[1], fanouts,
                                      kw.get("layered", False))
        loc = torch.full((B, ncap), -3, dtype=torch.int32, device=DEV)
        sr = dg.sample_group(off_d, idx_d, seeds_d, fanouts, rng_seed, batch_base=batch_base,
                             node_cap=ncap, edge_cap=ecap, cache_slot=slot, loc=loc, **kw)
        cap = max(int(sr.node_count.sum()), 1)
        out = dg.PackResult(packed=torch.empty((cap, R), dtype=torch.uint8, device=DEV),
                            packed_ids=torch.empty(cap, dtype=torch.int32, device=DEV),
                            packed_ptr=torch.empty(B + 1, dtype=torch.int64, device=DEV),
                            packed_ptr_host=np.zeros(B + 1, dtype=np.int64), loc=loc,
                            unique=torch.empty(cap, dtype=torch.int32, device=DEV), sizes={},
                            timing=None, row_bytes=R)
        pr = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True, out=out,
                           loc_pending=True)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    Y = []
    for b in range(seeds.shape[0]):
        n = int(sr.hop_ptr[b, -1])
        Y.append(dg.assemble_batch(cache, pr.chunk(b), pr.loc[b, :n], R, status=status))
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    return sr, pr, Y, cache


def compare_sampling(sr, ref, B):
    for b in range(B):
        n = int(sr.hop_ptr[b, -1])
        e = int(sr.edge_ptr[b, -1])
        assert np.array_equal(sr.hop_ptr[b], ref["hop_ptr"][b]), b
        assert np.array_equal(sr.edge_ptr[b], ref["edge_ptr"][b]), b
        assert np.array_equal(to_np(sr.nodes[b, :n]), ref["nodes"][b]), b
        assert np.array_equal(to_np(sr.edge_src[b, :e]), ref["edge_src"][b]), b
        assert np.array_equal(to_np(sr.edge_dst[b, :e]), ref["edge_dst"][b]), b


def compare_packing(pr, ref, B, full_rows=True):
    rows = ref["packed_rows"]
    assert pr.sizes["packed_rows"] == rows
    assert pr.sizes["unique_nodes"] == ref["unique_nodes"]
    assert pr.sizes["unique_packed"] == ref["unique_packed"]
    assert np.array_equal(pr.packed_ptr_host, ref["packed_ptr"])
    assert np.array_equal(to_np(pr.packed_ptr), ref["packed_ptr"])
    assert np.array_equal(to_np(pr.packed_ids[:rows]), ref["packed_ids"])
    assert np.array_equal(to_np(pr.unique[:ref["unique_nodes"]]), ref["unique"])
    for b in range(B):
        n = len(ref["loc"][b])
        assert np.array_equal(to_np(pr.loc[b, :n]), ref["loc"][b]), b
    if full_rows:
        assert np.array_equal(to_np(pr.packed[:rows]), ref["packed"])


def oracle_full(orc, off, idx, seeds, fanouts, rng_seed, feats, cache_slot, cache_nodes,
                batch_base=0, layered=False):
    X = to_np(feats)
    ref_s = orc.sample_group(to_np(off), to_np(idx), to_np(seeds), fanouts, rng_seed,
                             batch_base=batch_base, layered=layered)
    ref_p = orc.pack_group(X, to_np(cache_slot), ref_s["nodes"])
    R = X[0].nbytes
    cache = X[to_np(cache_nodes)] if cache_nodes.numel() else np.zeros((0,) + X.shape[1:], X.dtype)
    ref_y = []
    for b in range(len(ref_s["nodes"])):
        lo, hi = ref_p["packed_ptr"][b], ref_p["packed_ptr"][b + 1]
        ref_y.append(orc.assemble_batch(cache, ref_p["packed"][lo:hi], ref_p["loc"][b], R))
    return ref_s, ref_p, ref_y


def check_all(dg, orc, off, idx, seeds, fanouts, rng_seed, feats, cache_slot, cache_nodes,
              batch_base=0, sample_kw=None):
    sr, pr, Y, _ = run_path(dg, off, idx, seeds, fanouts, rng_seed, feats, cache_slot,
                            cache_nodes, batch_base, sample_kw)
    ref_s, ref_p, ref_y = oracle_full(orc, off, idx, seeds, fanouts, rng_seed, feats, cache_slot,
                                      cache_nodes, batch_base,
                                      layered=(sample_kw or {}).get("layered", False))
    B = seeds.shape[0]
    compare_sampling(sr, ref_s, B)
    compare_packing(pr, ref_p, B)
    X = to_np(feats).view(np.uint8).reshape(feats.shape[0], -1)
    for b in range(B):
        y = to_np(Y[b])
        assert np.array_equal(y, ref_y[b]), b
        assert np.array_equal(y, X[ref_s["nodes"][b]]), b        # closed form Y_b = X[nodes_b]
    return sr, pr


# ------------------------------------------------------------------ workloads
def test_tiny_workload_T(dg, orc):
    w = synth.make_workload("T")
    check_all(dg, orc, w.offsets, w.indices, w.seeds, list(w.cfg.fanouts), w.rng_seed, w.feats,
              w.cache_slot, w.cache_nodes)


def test_tiny_workload_T_layered(dg, orc):
    w = synth.make_workload("T")
    check_all(dg, orc, w.offsets, w.indices, w.seeds, list(w.cfg.fanouts), w.rng_seed, w.feats,
              w.cache_slot, w.cache_nodes, sample_kw={"layered": True})


@pytest.mark.parametrize("layered", [False, True])
def test_tiny_workload_T_direct_relabel(dg, orc, layered):
    w = synth.make_workload("T")
    check_all(dg, orc, w.offsets, w.indices, w.seeds, list(w.cfg.fanouts), w.rng_seed, w.feats,
              w.cache_slot, w.cache_nodes, sample_kw={"layered": layered, "direct": True})


@pytest.mark.parametrize("layered,direct", [(False, True), (True, True), (False, False)])
def test_tiny_workload_T_sample_and_pack_in_one_call(dg, orc, layered, direct):
    """dg_sample_pack_group: every output equals the oracle's, whether the
    last hop's compaction does packing's pass (direct table) or packing's own
    passes follow (hash relabelling)."""
    w = synth.make_workload("T")
    check_all(dg, orc, w.offsets, w.indices, w.seeds, list(w.cfg.fanouts), w.rng_seed, w.feats,
              w.cache_slot, w.cache_nodes,
              sample_kw={"layered": layered, "direct": direct, "handoff": "fused"})
    # which of the two ran: packing's own count pass times its ordering phase
    X, slot = w.feats.to(DEV), w.cache_slot.to(DEV)
    _, pr = dg.sample_pack_group(w.offsets.to(DEV), w.indices.to(DEV), w.seeds.to(DEV),
                                 list(w.cfg.fanouts), w.rng_seed, X, slot, timing=True,
                                 layered=layered, direct=direct)
    assert (pr.timing["order_ms"] == 0.0) == direct
    assert pr.timing["gather_ms"] > 0.0 and pr.timing["total_ms"] > 0.0


@pytest.mark.parametrize("direct", [False, True])
def test_tiny_workload_T_address_tables_from_sampling(dg, orc, direct):
    """Sampling writes the cached nodes' address-table entries as it lists
    them, and packing completes the others (DG_PACK_LOC_PENDING): every output
    equals the oracle's."""
    w = synth.make_workload("T")
    check_all(dg, orc, w.offsets, w.indices, w.seeds, list(w.cfg.fanouts), w.rng_seed, w.feats,
              w.cache_slot, w.cache_nodes, sample_kw={"direct": direct, "handoff": True})


def test_tiny_workload_T_is_deterministic(dg):
    w = synth.make_workload("T")
    a, pa, ya, _ = run_path(dg, w.offsets, w.indices, w.seeds, list(w.cfg.fanouts), w.rng_seed,
                            w.feats, w.cache_slot, w.cache_nodes)
    b, pb, yb, _ = run_path(dg, w.offsets, w.indices, w.seeds, list(w.cfg.fanouts), w.rng_seed,
                            w.feats, w.cache_slot, w.cache_nodes)
    for B in range(w.cfg.B):
        assert torch.equal(a.batch_nodes(B), b.batch_nodes(B))
        assert torch.equal(ya[B], yb[B])
    assert torch.equal(pa.packed, pb.packed)


def test_group_split_equals_whole(dg):
    w = synth.make_workload("T")
    fan = list(w.cfg.fanouts)
    whole = dg.sample_group(w.offsets.to(DEV), w.indices.to(DEV), w.seeds.to(DEV), fan,
                            w.rng_seed, batch_base=7)
    part0 = dg.sample_group(w.offsets.to(DEV), w.indices.to(DEV), w.seeds[:1].to(DEV), fan,
                            w.rng_seed, batch_base=7)
    part1 = dg.sample_group(w.offsets.to(DEV), w.indices.to(DEV), w.seeds[1:].contiguous().to(DEV),
                            fan, w.rng_seed, batch_base=8)
    parts = [(part0, 0)] + [(part1, i) for i in range(w.cfg.B - 1)]
    for b, (p, i) in enumerate(parts):
        assert torch.equal(whole.batch_nodes(b), p.batch_nodes(i))
        assert torch.equal(whole.batch_edges(b)[1], p.batch_edges(i)[1])


# ------------------------------------------------------------------ edge cases
def random_case(rnd, n, maxdeg):
    deg = [rnd.randint(0, min(maxdeg, n - 1)) for _ in range(n)]
    rows = [sorted(rnd.sample([u for u in range(n) if u != v], d)) for v, d in enumerate(deg)]
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(deg)
    idx = np.array([u for r in rows for u in r], dtype=np.int32)
    return torch.from_numpy(off), torch.from_numpy(idx)


CASES = [
    # (n, maxdeg, B, S, fanouts, row elems, dtype, cache share)
    (50, 8, 1, 1, [2, 2], 4, torch.float32, 0.0),
    (300, 30, 3, 7, [5, -1], 16, torch.float32, 0.2),
    (300, 60, 2, 5, [40, 3], 16, torch.float32, 0.5),          # f > register path
    (200, 12, 4, 9, [0, 3], 8, torch.float32, 0.1),            # f = 0 hop
    (500, 25, 64, 3, [4, 4, 4], 32, torch.float32, 0.05),      # B = 64
    (1000, 20, 5, 20, [10, 10, 10], 24, torch.float16, 0.3),   # 48-byte rows
    (400, 15, 3, 11, [15, 15], 3, torch.uint8, 0.0),           # 3-byte rows
    (400, 15, 3, 11, [7, 1], 5, torch.int16, 1.0),             # every node cached
    (777, 40, 7, 13, [-1, 2], 385, torch.float32, 0.02),       # 1540-byte rows
    (100, 99, 2, 4, [99, 99], 4, torch.float32, 0.0),          # f = d on full rows
    (2, 1, 2, 1, [1, 1, 1], 4, torch.float32, 0.0),            # tiny graph, cycles
    (64, 0, 3, 5, [3, 3], 4, torch.float32, 0.0),              # no edges at all
    (600, 20, 4, 8, [6, 6], 768, torch.float16, 0.1),          # 1536-byte rows (2 vectors/lane, 2nd half used)
    (600, 20, 4, 8, [6, 6], 512, torch.float32, 0.1),          # 2048-byte rows (2 vectors/lane)
    (600, 20, 4, 8, [6, 6], 1024, torch.float32, 0.1),         # 4096-byte rows (4 vectors/lane)
    (300, 20, 5, 6, [4, 0], 16, torch.float32, 0.2),           # f = 0 at the last hop
    (300, 20, 5, 6, [6], 16, torch.float32, 0.2),              # one hop (the last is the first)
    (300, 20, 5, 6, [], 16, torch.float32, 0.2),               # no hop: the seeds alone
    (300, 299, 64, 5, [-1, 2], 8, torch.float32, 0.3),         # every batch holds nearly every
                                                               # node: full 64-bit membership
                                                               # words, several 64-word chunks
                                                               # per wave in the write passes
]


@pytest.mark.parametrize("layered,direct,handoff", [
    (False, False, False), (True, False, False), (False, True, False), (True, True, False),
    (False, True, True), (True, False, True), (False, True, "fused"), (True, True, "fused"),
    (False, False, "fused")])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_edge_cases(dg, orc, case, layered, direct, handoff):
    n, maxdeg, B, S, fan, dim, dtype, share = CASES[case]
    rnd = random.Random(900 + case)
    off, idx = random_case(rnd, n, maxdeg) if maxdeg else (
        torch.zeros(n + 1, dtype=torch.int64), torch.zeros(0, dtype=torch.int32))
    seeds = torch.tensor([rnd.sample(range(n), S) for _ in range(B)], dtype=torch.int32)
    gen = torch.Generator().manual_seed(case)
    if dtype.is_floating_point:
        feats = torch.randn((n, dim), generator=gen).to(dtype)
    else:
        feats = torch.randint(0, 100, (n, dim), generator=gen).to(dtype)
    ncache = int(n * share)
    cache_nodes = torch.tensor(rnd.sample(range(n), ncache), dtype=torch.int64)
    slot = torch.full((n,), -1, dtype=torch.int32)
    slot[cache_nodes] = torch.arange(ncache, dtype=torch.int32)
    check_all(dg, orc, off, idx, seeds, fan, 12345 + case, feats, slot, cache_nodes,
              batch_base=case, sample_kw={"layered": layered, "direct": direct,
                                          "handoff": handoff})


def test_fig1_example_on_device(dg, orc):
    import json, os
    from conftest import GOLDEN
    fx = json.load(open(os.path.join(GOLDEN, "fig1_sampling.json")))
    n = fx["num_nodes"]
    off = np.zeros(n + 1, dtype=np.int64)
    idx = []
    for v in range(n):
        r = fx["rows"].get(str(v), [])
        idx += r
        off[v + 1] = off[v] + len(r)
    sr = dg.sample_group(torch.from_numpy(off).to(DEV), torch.tensor(idx, dtype=torch.int32,
                         device=DEV), torch.tensor(fx["seeds"], dtype=torch.int32, device=DEV),
                         fx["fanouts"], 0)
    assert to_np(sr.batch_nodes(0)).tolist() == fx["expect"]["nodes"]
    assert sr.hop_ptr[0].tolist() == fx["expect"]["hop_ptr"]


def test_membership_handoff_matches_standalone_pack(dg):
    """dg_sample_group's membership mask handed to dg_pack_group gives the
    same packing as rebuilding it from the lists; masks that disagree with the
    lists are rejected."""
    w = synth.make_workload("T")
    X, slot = w.feats.to(DEV), w.cache_slot.to(DEV)
    mem = torch.empty(w.cfg.n, dtype=torch.int64, device=DEV)
    sr = dg.sample_group(w.offsets.to(DEV), w.indices.to(DEV), w.seeds.to(DEV),
                         list(w.cfg.fanouts), w.rng_seed, membership=mem)
    # the mask is exactly the lists' membership
    want = torch.zeros(w.cfg.n, dtype=torch.int64)
    for b in range(w.cfg.B):
        want[sr.batch_nodes(b).long().cpu()] |= (1 << b)
    assert torch.equal(mem.cpu(), want)
    a = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True)
    b = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True, membership=mem)
    for key in ("packed_rows", "unique_nodes", "unique_packed"):
        assert a.sizes[key] == b.sizes[key]
    rows = a.sizes["packed_rows"]
    assert torch.equal(a.packed[:rows], b.packed[:rows])
    assert torch.equal(a.packed_ids[:rows], b.packed_ids[:rows])
    assert torch.equal(a.unique, b.unique)
    for bb in range(w.cfg.B):
        n = int(sr.hop_ptr[bb, -1])
        assert torch.equal(a.loc[bb, :n], b.loc[bb, :n])
    # a list entry missing from the mask
    bad = mem.clone()
    u = int(sr.batch_nodes(2)[5])
    bad[u] &= ~(1 << 2)
    with pytest.raises(dg.DGError):
        dg.pack_group(X, slot, sr.nodes, sr.node_count, membership=bad)
    # an extra (node, batch) pair in the mask
    bad = mem.clone()
    free = int((mem == 0).nonzero()[0])
    bad[free] = 1
    with pytest.raises(dg.DGError):
        dg.pack_group(X, slot, sr.nodes, sr.node_count, membership=bad)


def test_assemble_batches_matches_per_batch_calls(dg):
    """The group helper issues the same per-batch library call; outputs equal
    dg_assemble_batch's, batch by batch, and out-of-range loc is flagged."""
    w = synth.make_workload("T")
    X, slot = w.feats.to(DEV), w.cache_slot.to(DEV)
    sr = dg.sample_group(w.offsets.to(DEV), w.indices.to(DEV), w.seeds.to(DEV),
                         list(w.cfg.fanouts), w.rng_seed)
    pr = dg.pack_group(X, slot, sr.nodes, sr.node_count)
    cache = X.index_select(0, w.cache_nodes.to(DEV))
    R = pr.row_bytes
    counts = sr.node_count
    outs = [torch.full((int(counts.max()), R), 0xAB, dtype=torch.uint8, device=DEV)
            for _ in range(len(counts))]
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dg.assemble_batches(cache, pr, counts, outs, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for b, n in enumerate(counts):
        ref = dg.assemble_batch(cache, pr.chunk(b), pr.loc[b, :int(n)], R)
        assert torch.equal(outs[b][:int(n)], ref), b
    with pytest.raises(ValueError):
        dg.assemble_batches(cache, pr, counts, [outs[0][:1]])


def buffer_test_group(dg, group, dim):
    """(cache, packing result, counts) of one sampled and packed group: workload
    T (4 mini-batches), or a group of 20 mini-batches on a small random graph,
    so that launches of eight consecutive mini-batches and a shorter last one
    occur."""
    gen = torch.Generator().manual_seed(dim)
    if group == "T":
        w = synth.make_workload("T")
        X = torch.randn((w.cfg.n, dim), generator=gen).to(DEV)
        slot = w.cache_slot.to(DEV)
        sr = dg.sample_group(w.offsets.to(DEV), w.indices.to(DEV), w.seeds.to(DEV),
                             list(w.cfg.fanouts), w.rng_seed)
        cache_nodes = w.cache_nodes.to(DEV)
    else:
        n, B, S = 2000, 20, 8
        rnd = random.Random(4242)
        off, idx = random_case(rnd, n, 20)
        seeds = torch.tensor([rnd.sample(range(n), S) for _ in range(B)], dtype=torch.int32)
        X = torch.randn((n, dim), generator=gen).to(DEV)
        cache_nodes = torch.tensor(rnd.sample(range(n), n // 10), dtype=torch.int64)
        slot = torch.full((n,), -1, dtype=torch.int32)
        slot[cache_nodes] = torch.arange(n // 10, dtype=torch.int32)
        slot, cache_nodes = slot.to(DEV), cache_nodes.to(DEV)
        sr = dg.sample_group(off.to(DEV), idx.to(DEV), seeds.to(DEV), [5, 5], 99)
    pr = dg.pack_group(X, slot, sr.nodes, sr.node_count)
    return X.index_select(0, cache_nodes), pr, sr.node_count


@pytest.mark.parametrize("group,dim", [("T", 16), ("T", 128), ("T", 384), ("T", 512),
                                       ("T", 1024), ("wide", 16), ("wide", 512)])
@pytest.mark.parametrize("outs_kind", ["one", "two", "same_twice", "eight", "nine", "all"])
def test_assemble_batches_output_buffers(dg, group, dim, outs_kind):
    """Batches whose output buffers are distinct may share a launch; the
    result must still be that of the per-batch calls made in batch order, on
    every 16-byte row shape (64 B to 4 KiB rows): with one buffer (each batch
    overwrites the last), two, eight or nine buffers (batch b in buffer
    b % count), the same buffer given twice (no sharing possible), and a
    buffer per batch; with 4 mini-batches and with 20 (launches of eight and
    a shorter last one)."""
    cache, pr, counts = buffer_test_group(dg, group, dim)
    R = pr.row_bytes
    B, nmax = len(counts), int(counts.max())
    refs = [dg.assemble_batch(cache, pr.chunk(b), pr.loc[b, :int(counts[b])], R).clone()
            for b in range(B)]
    one = torch.full((nmax, R), 0xAB, dtype=torch.uint8, device=DEV)
    if outs_kind == "same_twice":
        outs = [one, one]
    else:
        count = {"one": 1, "two": 2, "eight": 8, "nine": 9, "all": B}[outs_kind]
        outs = [one] + [torch.full((nmax, R), 0xAB, dtype=torch.uint8, device=DEV)
                        for _ in range(count - 1)]
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dg.assemble_batches(cache, pr, counts, outs, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    # each buffer holds the last batch written to it, over what earlier batches left
    expect = [torch.full((nmax, R), 0xAB, dtype=torch.uint8, device=DEV) for _ in outs]
    for b in range(B):
        k = b % len(outs)
        tgt = expect[0] if outs_kind == "same_twice" else expect[k]
        tgt[:int(counts[b])] = refs[b]
    for k, o in enumerate(outs):
        want = expect[0] if outs_kind == "same_twice" else expect[k]
        assert torch.equal(o, want), k


@pytest.mark.parametrize("layered,direct,handoff", [(False, False, False), (True, True, False),
                                                    (False, True, True), (False, True, "fused")])
def test_sparse_hops_on_a_large_graph(dg, orc, layered, direct, handoff):
    """A small frontier on a large graph: every hop's edges reach only a small
    share of the nodes, so the sampler lists new nodes from the 8-node mask
    lines its draws touched (the count pass skips the others)."""
    n = 200_000
    off, idx = synth.uniform_graph(n, 0, 6, seed=31)
    off, idx = torch.from_numpy(off), torch.from_numpy(idx)
    rnd = random.Random(4242)
    seeds = torch.tensor([rnd.sample(range(n), 16) for _ in range(4)], dtype=torch.int32)
    gen = torch.Generator().manual_seed(7)
    feats = torch.randn((n, 4), generator=gen)
    ncache = n // 10
    cache_nodes = torch.tensor(rnd.sample(range(n), ncache), dtype=torch.int64)
    slot = torch.full((n,), -1, dtype=torch.int32)
    slot[cache_nodes] = torch.arange(ncache, dtype=torch.int32)
    check_all(dg, orc, off, idx, seeds, [3, 3, 2], 99, feats, slot, cache_nodes, batch_base=5,
              sample_kw={"layered": layered, "direct": direct, "handoff": handoff})


def test_assemble_batches_in_a_hip_graph(dg):
    """dg_assemble_batches captured into a HIP graph (kernel launches only, no
    memset) replays to the eager result, replay after replay, with eager work
    in between."""
    w = synth.make_workload("T")
    X, slot = w.feats.to(DEV), w.cache_slot.to(DEV)
    sr = dg.sample_group(w.offsets.to(DEV), w.indices.to(DEV), w.seeds.to(DEV),
                         list(w.cfg.fanouts), w.rng_seed)
    pr = dg.pack_group(X, slot, sr.nodes, sr.node_count)
    cache = X.index_select(0, w.cache_nodes.to(DEV))
    R = pr.row_bytes
    counts = sr.node_count
    nmax = int(counts.max())
    ref = [torch.empty((nmax, R), dtype=torch.uint8, device=DEV) for _ in range(len(counts))]
    dg.assemble_batches(cache, pr, counts, ref)
    outs = [torch.empty((nmax, R), dtype=torch.uint8, device=DEV) for _ in range(len(counts))]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm up on the capture stream
        dg.assemble_batches(cache, pr, counts, outs, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dg.assemble_batches(cache, pr, counts, outs, stream=torch.cuda.current_stream())
    for rep in range(3):
        for o in outs:
            o.fill_(rep + 1)
        dg.assemble_batch(cache, pr.chunk(0), pr.loc[0, :int(counts[0])], R)  # eager work
        g.replay()
        torch.cuda.synchronize()
        for b, n in enumerate(counts):
            assert torch.equal(outs[b][:int(n)], ref[b][:int(n)]), (rep, b)


@pytest.mark.parametrize("name", ["T", "M1"])
def test_pack_rows_on_a_second_stream(dg, name):
    """DG_PACK_ROWS_STREAM: the row copy left queued on a second stream, and the
    assembly queued behind it on that stream without a host wait, give the
    outputs of the ordinary call."""
    w = synth.make_workload(name, device=DEV)
    X, slot = w.feats, w.cache_slot
    sr = dg.sample_group(w.offsets, w.indices, w.seeds, list(w.cfg.fanouts), w.rng_seed)
    counts = sr.node_count
    ref = dg.pack_group(X, slot, sr.nodes, counts, with_unique=True)
    R = ref.row_bytes
    out = dg.pack_group(X, slot, sr.nodes, counts, with_unique=True)  # same-size buffers
    out.packed.zero_()
    nmax = int(counts.max())
    ys = [torch.full((nmax, R), 0xEE, dtype=torch.uint8, device=DEV) for _ in counts]
    side = torch.cuda.Stream(device=DEV)
    torch.cuda.synchronize()
    for rep in range(2):  # twice on the same buffers and workspace
        ws = torch.empty(dg._L.dg_pack_workspace_bytes(w.cfg.n, w.cfg.B, int(counts.sum())),
                         dtype=torch.uint8, device=DEV)
        pr = dg.pack_group(X, slot, sr.nodes, counts, with_unique=True, out=out, workspace=ws,
                           rows_stream=side)
        done = torch.cuda.Event()
        done.record(torch.cuda.current_stream())
        side.wait_event(done)  # the address tables are on the caller's stream
        dg.assemble_batches(w.cache, pr, counts, ys, stream=side)
        side.synchronize()
        rows = ref.sizes["packed_rows"]
        assert pr.sizes == ref.sizes
        assert torch.equal(pr.packed[:rows], ref.packed[:rows]), rep
        assert torch.equal(pr.packed_ids[:rows], ref.packed_ids[:rows])
        for b, n in enumerate(counts):
            n = int(n)
            assert torch.equal(pr.loc[b, :n], ref.loc[b, :n]), b
            assert torch.equal(ys[b][:n], X.index_select(0, sr.nodes[b, :n].long())
                               .view(torch.uint8).reshape(n, R)), b
        del ws


def layered_star_graph(n, n_seed, seed_deg, n_mid, mid_deg, seed=0):
    """CSR where nodes [0, n_seed) point to `seed_deg` random nodes of the middle
    range [n_seed, n_seed + n_mid), middle nodes to `mid_deg` random nodes of
    [0, n), and every other node to none: a two-hop sample reaches a few
    thousand middle nodes, then hundreds of thousands of new nodes."""
    rng = np.random.default_rng(seed)
    deg = np.zeros(n, dtype=np.int64)
    deg[:n_seed] = seed_deg
    deg[n_seed:n_seed + n_mid] = mid_deg
    off = np.zeros(n + 1, dtype=np.int64)
    off[1:] = np.cumsum(deg)
    rows = []
    for v in range(n_seed + n_mid):
        if v < n_seed:
            r = rng.choice(np.arange(n_seed, n_seed + n_mid), seed_deg, replace=False)
        else:
            r = rng.choice(n, mid_deg + 1, replace=False)
            r = r[r != v][:mid_deg]
        rows.append(np.sort(r))
    return torch.from_numpy(off), torch.from_numpy(np.concatenate(rows).astype(np.int32))


@pytest.mark.parametrize("last_fanout", [150, 260])
def test_last_hop_segments_of_a_few_hundred_thousand_nodes(dg, orc, last_fanout):
    """The last hop lists about 0.4M (fan-out 150) and 0.7M (260) new nodes in
    one mini-batch, beyond the shortest block length of the last hop's search
    (2^18 nodes), so both longer block lengths run; and its edges into nodes of
    the first hop still go through the table.  Bit-exact against the oracle,
    with and without the cached nodes' address tables from sampling."""
    n, n_seed, n_mid = 4_000_000, 4096, 3000
    off, idx = layered_star_graph(n, n_seed, 20, n_mid, 300, seed=last_fanout)
    seeds = torch.stack([torch.arange(0, 2048, dtype=torch.int32),
                         torch.arange(2048, 4096, dtype=torch.int32)])
    gen = torch.Generator().manual_seed(3)
    feats = torch.randn((n, 4), generator=gen)
    rnd = random.Random(last_fanout)
    ncache = n // 20
    cache_nodes = torch.tensor(rnd.sample(range(n), ncache), dtype=torch.int64)
    slot = torch.full((n,), -1, dtype=torch.int32)
    slot[cache_nodes] = torch.arange(ncache, dtype=torch.int32)
    for handoff in (False, True, "fused"):
        sr, _ = check_all(dg, orc, off, idx, seeds, [5, last_fanout], 77, feats, slot,
                          cache_nodes, sample_kw={"direct": True, "handoff": handoff})
        m = [int(sr.hop_ptr[b, -1] - sr.hop_ptr[b, -2]) for b in range(2)]
        assert max(m) > (1 << 18), m  # beyond the shortest block length


@pytest.mark.parametrize("direct", [False, True])
def test_unaligned_list_outputs(dg, direct):
    """Node lists, address tables and packed IDs handed over at 4-byte (not
    16-byte) alignment give the outputs of aligned buffers, and nothing is
    written before them."""
    w = synth.make_workload("T")
    off, idx, seeds = w.offsets.to(DEV), w.indices.to(DEV), w.seeds.to(DEV)
    X, slot = w.feats.to(DEV), w.cache_slot.to(DEV)
    fan = list(w.cfg.fanouts)
    B = w.cfg.B
    ncap, ecap = dg.sample_bounds(w.cfg.n, w.num_edges, w.cfg.S, fan)
    ref = dg.sample_group(off, idx, seeds, fan, w.rng_seed, direct=direct, node_cap=ncap,
                          edge_cap=ecap)
    ref_p = dg.pack_group(X, slot, ref.nodes, ref.node_count, with_unique=True)
    big = torch.full((B * ncap + 1,), -9, dtype=torch.int32, device=DEV)
    nodes = big[1:].view(B, ncap)  # one element past a 16-byte boundary
    assert nodes.data_ptr() % 16 == 4
    out = dg.SampleResult(nodes=nodes, hop_ptr=np.zeros((B, len(fan) + 2), dtype=np.int64),
                          edge_src=torch.empty((B, ecap), dtype=torch.int32, device=DEV),
                          edge_dst=torch.empty((B, ecap), dtype=torch.int32, device=DEV),
                          edge_ptr=np.zeros((B, len(fan) + 1), dtype=np.int64), sizes={},
                          timing=None)
    bigl = torch.full((B * ncap + 1,), -9, dtype=torch.int32, device=DEV)
    loc = bigl[1:].view(B, ncap)
    sr = dg.sample_group(off, idx, seeds, fan, w.rng_seed, direct=direct, out=out,
                         cache_slot=slot, loc=loc)
    rows = ref_p.sizes["packed_rows"]
    bigp = torch.full((rows + 1,), -9, dtype=torch.int32, device=DEV)
    po = dg.PackResult(packed=torch.empty((rows, ref_p.row_bytes), dtype=torch.uint8, device=DEV),
                       packed_ids=bigp[1:], packed_ptr=torch.empty(B + 1, dtype=torch.int64,
                                                                   device=DEV),
                       packed_ptr_host=np.zeros(B + 1, dtype=np.int64), loc=loc,
                       unique=torch.empty(ref_p.unique.numel(), dtype=torch.int32, device=DEV),
                       sizes={}, timing=None, row_bytes=ref_p.row_bytes)
    pr = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True, out=po,
                       loc_pending=True)
    torch.cuda.synchronize()
    assert int(big[0]) == -9 and int(bigl[0]) == -9 and int(bigp[0]) == -9
    assert np.array_equal(sr.hop_ptr, ref.hop_ptr) and np.array_equal(sr.edge_ptr, ref.edge_ptr)
    for b in range(B):
        n, e = int(ref.hop_ptr[b, -1]), int(ref.edge_ptr[b, -1])
        assert torch.equal(sr.nodes[b, :n], ref.nodes[b, :n]), b
        assert torch.equal(sr.edge_dst[b, :e], ref.edge_dst[b, :e]), b
        assert torch.equal(pr.loc[b, :n], ref_p.loc[b, :n]), b
    assert torch.equal(pr.packed_ids[:rows], ref_p.packed_ids[:rows])
    assert torch.equal(pr.packed[:rows], ref_p.packed[:rows])
