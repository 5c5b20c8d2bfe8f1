"""Parity on the named workloads, in the launch configuration bench.py times:
the sampler's membership mask handed to the packer, the mask-clearing flags
(two groups in a row on the same membership buffer and workspaces, the second
sampling call told that the state is clear, and the second also taking the
cached nodes' address-table entries from sampling), and packing's row copy
queued on a second stream with the assembly behind it.  A third run samples
and packs the group in one dg_sample_pack_group call.

Every workload compares, for every mini-batch of the group, the sampled node
list, hop bounds, edge lists and edge bounds with the oracle's (one oracle run
over the whole group, split over host threads by runs of batches; each draw is
keyed by its global batch number, so the split changes nothing), and every
packing table of the whole group (U, P_b order, packed_ptr, address tables)
with the oracle's packing of those same lists.  M1 also compares feature rows
with the oracle's own copies; at full size (L100, W120, H65 at every cache
share) every packed and every assembled row is checked on the device against
an independent library gather (torch.index_select) of the feature table.
L100, H65 and M1 relabel through the direct [N][B] table (as bench.py does);
W120 runs the three through the hash table, then once more in one call with the
direct table, as bench.py runs it.  L100 and M1 are also sampled with layer-wise
frontiers and compared with the oracle batch by batch."""
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


def rows_equal(a: torch.Tensor, b: torch.Tensor) -> bool:
    return torch.equal(a.view(torch.uint8).reshape(a.shape[0], -1),
                       b.contiguous().view(torch.uint8).reshape(b.shape[0], -1))


def check_rows_on_device(X, ids, got, chunk=1 << 20):
    """got[i] == X[ids[i]] bitwise, in chunks."""
    for lo in range(0, ids.numel(), chunk):
        hi = min(ids.numel(), lo + chunk)
        ref = X.index_select(0, ids[lo:hi].long())
        assert rows_equal(got[lo:hi], ref), (lo, hi)


def bench_path(dg, w, fan, mem, ws_s, ws_p, direct, entry_clear, out=None, pack_out=None):
    """One group as bench.py runs it: sampling with the clearing flags, packing
    that clears the mask and leaves its row copy on a second stream.  With
    pack_out (a packing output set of this group's sizes, its address table
    laid out as the node lists), sampling also writes the cached nodes'
    address-table entries into it and packing completes the others."""
    sr = dg.sample_group(w.offsets, w.indices, w.seeds, fan, w.rng_seed, membership=mem,
                         workspace=ws_s, direct=direct, exit_clear=True,
                         entry_clear=entry_clear, out=out,
                         cache_slot=w.cache_slot if pack_out is not None else None,
                         loc=pack_out.loc if pack_out is not None else None)
    counts = sr.node_count.copy()
    side = torch.cuda.Stream(device=DEV)
    pr = dg.pack_group(w.feats, w.cache_slot, sr.nodes, counts, with_unique=True, membership=mem,
                       workspace=ws_p, clear_membership=True, rows_stream=side, out=pack_out,
                       loc_pending=pack_out is not None)
    side.synchronize()
    torch.cuda.synchronize()
    return sr, counts, pr


def oracle_sample(orc, w, layered=False):
    """The oracle's sampling of the workload's whole group, every batch."""
    return orc.sample_group(w.offsets.cpu().numpy(), w.indices.cpu().numpy(),
                            w.seeds.cpu().numpy(), list(w.cfg.fanouts), w.rng_seed,
                            layered=layered, threads=orc.host_threads())


def compare_samples(sr, ref, B):
    for b in range(B):
        n, e = int(sr.hop_ptr[b, -1]), int(sr.edge_ptr[b, -1])
        assert np.array_equal(sr.hop_ptr[b], ref["hop_ptr"][b]), b
        assert np.array_equal(sr.edge_ptr[b], ref["edge_ptr"][b]), b
        assert np.array_equal(sr.nodes[b, :n].cpu().numpy(), ref["nodes"][b]), b
        assert np.array_equal(sr.edge_src[b, :e].cpu().numpy(), ref["edge_src"][b]), b
        assert np.array_equal(sr.edge_dst[b, :e].cpu().numpy(), ref["edge_dst"][b]), b


def run_and_check(dg, orc, w, ref, direct=True):
    """ref: the oracle's sampling of the whole group (oracle_sample)."""
    cfg = w.cfg
    fan = list(cfg.fanouts)
    R = cfg.row_bytes
    mem = torch.full((cfg.n,), -1, dtype=torch.int64, device=DEV)  # garbage on entry
    node_cap, edge_cap = dg.sample_bounds(cfg.n, w.num_edges, cfg.S, fan)
    ws_s = torch.empty(dg._L.dg_sample_workspace_bytes(cfg.n, cfg.B, node_cap, edge_cap,
                                                       dg.sample_flags(direct=direct)),
                       dtype=torch.uint8, device=DEV)
    ws_p = torch.empty(dg._L.dg_pack_workspace_bytes(cfg.n, cfg.B, cfg.B * node_cap),
                       dtype=torch.uint8, device=DEV)
    sr, counts, pr = bench_path(dg, w, fan, mem, ws_s, ws_p, direct, entry_clear=False)
    assert int(mem.count_nonzero()) == 0
    print(f"[{cfg.name}] nodes {sr.sizes['total_nodes']:,} edges {sr.sizes['total_edges']:,} "
          f"packed {pr.sizes['packed_rows']:,} U {pr.sizes['unique_nodes']:,}", flush=True)

    # sampling: every batch against the oracle
    compare_samples(sr, ref, cfg.B)

    # packing tables of the whole group: the oracle's packing of its own lists
    # (equal to the device's, as just checked)
    refp = orc.pack_group(None, w.cache_slot.cpu().numpy(), ref["nodes"], rows=False,
                          row_bytes=R)
    rows = refp["packed_rows"]
    assert pr.sizes["packed_rows"] == rows
    assert pr.sizes["unique_nodes"] == refp["unique_nodes"]
    assert pr.sizes["unique_packed"] == refp["unique_packed"]
    assert np.array_equal(pr.packed_ptr_host, refp["packed_ptr"])
    assert np.array_equal(pr.packed_ids[:rows].cpu().numpy(), refp["packed_ids"])
    assert np.array_equal(pr.unique[:refp["unique_nodes"]].cpu().numpy(), refp["unique"])
    for b in range(cfg.B):
        assert np.array_equal(pr.loc[b, :int(counts[b])].cpu().numpy(), refp["loc"][b]), b
    # rows
    check_rows_on_device(w.feats, pr.packed_ids[:rows], pr.packed[:rows].view(w.feats.dtype)
                         .reshape(rows, -1))
    out = torch.empty((int(counts.max()), R), dtype=torch.uint8, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    for b in range(cfg.B):
        n = int(counts[b])
        y = dg.assemble_batch(w.cache, pr.chunk(b), pr.loc[b, :n], R, out=out, status=status)
        check_rows_on_device(w.feats, sr.nodes[b, :n], y[:n].view(w.feats.dtype).reshape(n, -1))
    assert int(status.item()) == 0

    # a second group on the same buffers, told that the state is clear, with
    # the address tables of cached nodes written by sampling (into the first
    # call's packing set, garbage first) and completed by packing: the same
    # seeds give the same outputs
    keep = (sr.nodes.clone(), sr.edge_src.clone(), sr.edge_dst.clone(), sr.hop_ptr.copy(),
            sr.edge_ptr.copy(), pr.packed_ids[:rows].clone(), pr.loc.clone(),
            pr.packed[:rows].clone())
    pr.loc.fill_(-3)
    pr.packed[:rows].zero_()
    sr2, counts2, pr2 = bench_path(dg, w, fan, mem, ws_s, ws_p, direct, entry_clear=True,
                                   pack_out=pr)
    assert np.array_equal(counts2, counts) and np.array_equal(sr2.hop_ptr, keep[3])
    assert np.array_equal(sr2.edge_ptr, keep[4])
    for b in range(cfg.B):
        n, e = int(counts[b]), int(keep[4][b, -1])
        assert torch.equal(sr2.nodes[b, :n], keep[0][b, :n]), b
        assert torch.equal(sr2.edge_src[b, :e], keep[1][b, :e]), b
        assert torch.equal(sr2.edge_dst[b, :e], keep[2][b, :e]), b
        assert torch.equal(pr2.loc[b, :n], keep[6][b, :n]), b
    assert torch.equal(pr2.packed_ids[:rows], keep[5])
    assert torch.equal(pr2.packed[:rows], keep[7])
    assert int(mem.count_nonzero()) == 0

    # a third time in one dg_sample_pack_group call (with the direct table its
    # last hop's compaction does packing's pass; with the hash table packing's
    # own passes follow), still told that the state is clear, every output
    # overwritten with garbage first
    for t in (sr2.nodes, sr2.edge_src, sr2.edge_dst, pr2.packed_ids, pr2.unique):
        t.fill_(-7)
    pr2.loc.fill_(-3)
    pr2.packed[:rows].zero_()
    ws_f = torch.empty(dg._L.dg_sample_pack_workspace_bytes(cfg.n, cfg.B, node_cap),
                       dtype=torch.uint8, device=DEV)
    side = torch.cuda.Stream(device=DEV)
    sr3, pr3 = dg.sample_pack_group(w.offsets, w.indices, w.seeds, fan, w.rng_seed, w.feats,
                                    w.cache_slot, out=sr2, pack_out=pr2, workspace=ws_s,
                                    pack_workspace=ws_f, rows_stream=side, membership=mem,
                                    direct=direct, exit_clear=True, entry_clear=True)
    side.synchronize()
    torch.cuda.synchronize()
    assert np.array_equal(sr3.hop_ptr, keep[3]) and np.array_equal(sr3.edge_ptr, keep[4])
    for b in range(cfg.B):
        n, e = int(counts[b]), int(keep[4][b, -1])
        assert torch.equal(sr3.nodes[b, :n], keep[0][b, :n]), b
        assert torch.equal(sr3.edge_src[b, :e], keep[1][b, :e]), b
        assert torch.equal(sr3.edge_dst[b, :e], keep[2][b, :e]), b
        assert torch.equal(pr3.loc[b, :n], keep[6][b, :n]), b
    assert pr3.sizes["packed_rows"] == rows
    assert pr3.sizes["unique_nodes"] == refp["unique_nodes"]
    assert np.array_equal(pr3.packed_ptr_host, refp["packed_ptr"])
    assert np.array_equal(pr3.packed_ptr.cpu().numpy(), refp["packed_ptr"])
    assert torch.equal(pr3.packed_ids[:rows], keep[5])
    assert np.array_equal(pr3.unique[:refp["unique_nodes"]].cpu().numpy(), refp["unique"])
    assert torch.equal(pr3.packed[:rows], keep[7])
    assert int(mem.count_nonzero()) == 0
    print(f"[{cfg.name}] one-call sampling and packing equal", flush=True)
    return sr3, pr3


def one_call_check(dg, orc, w, ref):
    """The group in one dg_sample_pack_group call with the direct table (so
    that the last hop's compaction does packing's pass), the row copy on a
    second stream, garbage in every output and in the membership words (the
    call told nothing about their state): every batch's sample against the
    oracle's (ref), the packing tables against the oracle's packing, and every
    packed and assembled row against a library gather of the feature table."""
    cfg = w.cfg
    fan = list(cfg.fanouts)
    R = cfg.row_bytes
    node_cap, edge_cap = dg.sample_bounds(cfg.n, w.num_edges, cfg.S, fan)
    mem = torch.full((cfg.n,), -1, dtype=torch.int64, device=DEV)
    refp = orc.pack_group(None, w.cache_slot.cpu().numpy(), ref["nodes"], rows=False,
                          row_bytes=R)
    rows, nu = refp["packed_rows"], refp["unique_nodes"]
    out = dg.PackResult(packed=torch.zeros((rows, R), dtype=torch.uint8, device=DEV),
                        packed_ids=torch.full((rows,), -7, dtype=torch.int32, device=DEV),
                        packed_ptr=torch.full((cfg.B + 1,), -7, dtype=torch.int64, device=DEV),
                        packed_ptr_host=np.zeros(cfg.B + 1, dtype=np.int64),
                        loc=torch.full((cfg.B, node_cap), -3, dtype=torch.int32, device=DEV),
                        unique=torch.full((nu,), -7, dtype=torch.int32, device=DEV), sizes={},
                        timing=None, row_bytes=R)
    side = torch.cuda.Stream(device=DEV)
    sr, pr = dg.sample_pack_group(w.offsets, w.indices, w.seeds, fan, w.rng_seed, w.feats,
                                  w.cache_slot, node_cap=node_cap, edge_cap=edge_cap,
                                  pack_out=out, rows_stream=side, membership=mem, direct=True,
                                  exit_clear=True)
    side.synchronize()
    torch.cuda.synchronize()
    assert int(mem.count_nonzero()) == 0
    compare_samples(sr, ref, cfg.B)
    assert pr.sizes["packed_rows"] == rows and pr.sizes["unique_nodes"] == nu
    assert pr.sizes["unique_packed"] == refp["unique_packed"]
    assert np.array_equal(pr.packed_ptr_host, refp["packed_ptr"])
    assert np.array_equal(pr.packed_ptr.cpu().numpy(), refp["packed_ptr"])
    assert np.array_equal(pr.packed_ids.cpu().numpy(), refp["packed_ids"])
    assert np.array_equal(pr.unique.cpu().numpy(), refp["unique"])
    counts = sr.node_count
    for b in range(cfg.B):
        assert np.array_equal(pr.loc[b, :int(counts[b])].cpu().numpy(), refp["loc"][b]), b
    check_rows_on_device(w.feats, pr.packed_ids, pr.packed.view(w.feats.dtype).reshape(rows, -1))
    y = torch.empty((int(counts.max()), R), dtype=torch.uint8, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    for b in range(cfg.B):
        n = int(counts[b])
        dg.assemble_batch(w.cache, pr.chunk(b), pr.loc[b, :n], R, out=y, status=status)
        check_rows_on_device(w.feats, sr.nodes[b, :n], y[:n].view(w.feats.dtype).reshape(n, -1))
    assert int(status.item()) == 0
    print(f"[{cfg.name}] one call with the direct table equal to the oracle", flush=True)


def test_workload_M1_full(dg, orc):
    w = synth.make_workload("M1", device=DEV)
    sr, pr = run_and_check(dg, orc, w, oracle_sample(orc, w))
    # every row also against the oracle's own copies on a few batches
    X = w.feats.cpu().numpy()
    lists = [sr.nodes[b, :int(sr.hop_ptr[b, -1])].cpu().numpy() for b in (0, 1)]
    refp = orc.pack_group(X, w.cache_slot.cpu().numpy(), lists)
    cache = w.cache.cpu().numpy()
    for b in (0, 1):
        lo, hi = refp["packed_ptr"][b], refp["packed_ptr"][b + 1]
        y_ref = orc.assemble_batch(cache, refp["packed"][lo:hi], refp["loc"][b], w.cfg.row_bytes)
        n = len(lists[b])
        y = dg.assemble_batch(w.cache, pr.chunk(b), pr.loc[b, :n], w.cfg.row_bytes)
        assert np.array_equal(y.cpu().numpy(), y_ref)


def big(name, cache_pct=None):
    w = synth.make_workload(name, device=DEV, cache_pct=cache_pct)
    torch.cuda.synchronize()
    return w


def layered_check(dg, orc, w):
    """Layer-wise frontiers (every node so far samples at each hop), every
    batch against the oracle, direct relabelling table."""
    fan = list(w.cfg.fanouts)
    sr = dg.sample_group(w.offsets, w.indices, w.seeds, fan, w.rng_seed, layered=True,
                         direct=True)
    print(f"[{w.cfg.name} layered] nodes {sr.sizes['total_nodes']:,} "
          f"edges {sr.sizes['total_edges']:,}", flush=True)
    compare_samples(sr, oracle_sample(orc, w, layered=True), w.cfg.B)


@pytest.mark.big
@pytest.mark.timeout(900)
def test_workload_L100(dg, orc):
    w = big("L100")
    run_and_check(dg, orc, w, oracle_sample(orc, w))
    torch.cuda.empty_cache()
    layered_check(dg, orc, w)


@pytest.mark.big
@pytest.mark.timeout(900)
def test_workload_W120(dg, orc):
    w = big("W120")
    ref = oracle_sample(orc, w)
    run_and_check(dg, orc, w, ref, direct=False)
    torch.cuda.empty_cache()
    # the benchmark's configuration for W120: direct table, one call
    one_call_check(dg, orc, w, ref)


@pytest.mark.big
@pytest.mark.timeout(1200)
def test_workload_H65_cache_sweep(dg, orc):
    w = big("H65", cache_pct=0)
    ref = oracle_sample(orc, w)  # sampling does not depend on the cache
    for pct in synth.CONFIGS["H65"].cache_pct:
        synth.set_cache(w, pct)
        print(f"[H65] cache {pct}%", flush=True)
        run_and_check(dg, orc, w, ref)
        torch.cuda.empty_cache()


def test_workload_M1_layered_full(dg, orc):
    """Layer-wise frontiers at M1 scale, every batch against the oracle."""
    layered_check(dg, orc, synth.make_workload("M1", device=DEV))


def test_workload_M1_relabelling_tables_agree(dg):
    """The hash-table and direct-table relabelling give identical outputs."""
    w = synth.make_workload("M1", device=DEV)
    fan = list(w.cfg.fanouts)
    a = dg.sample_group(w.offsets, w.indices, w.seeds, fan, w.rng_seed, direct=False)
    b = dg.sample_group(w.offsets, w.indices, w.seeds, fan, w.rng_seed, direct=True)
    assert np.array_equal(a.hop_ptr, b.hop_ptr) and np.array_equal(a.edge_ptr, b.edge_ptr)
    for bb in range(w.cfg.B):
        n, e = int(a.hop_ptr[bb, -1]), int(a.edge_ptr[bb, -1])
        assert torch.equal(a.nodes[bb, :n], b.nodes[bb, :n])
        assert torch.equal(a.edge_src[bb, :e], b.edge_src[bb, :e])
        assert torch.equal(a.edge_dst[bb, :e], b.edge_dst[bb, :e])
