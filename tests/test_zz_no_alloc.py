"""dg_pack_group_noalloc (the allocation-free packing entry point) against
dg_pack_group on the same inputs, through the C ABI: every output equal, on
calls in a row that share the library's fixed scratch, each later one
smaller (fewer mini-batches, then a smaller graph), with and without a given
membership mask; and the scratch limit reported before any work."""
import ctypes

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


def packed_out(dg, ref, R):
    """Output buffers of ref's sizes, filled with garbage."""
    B, stride = ref.loc.shape
    rows = max(ref.sizes["packed_rows"], 1)
    nu = max(ref.sizes["unique_nodes"], 1)
    return dg.PackResult(
        packed=torch.full((rows, R), 0xAB, dtype=torch.uint8, device=DEV),
        packed_ids=torch.full((rows,), -7, dtype=torch.int32, device=DEV),
        packed_ptr=torch.full((B + 1,), -7, dtype=torch.int64, device=DEV),
        packed_ptr_host=np.full(B + 1, -7, dtype=np.int64),
        loc=torch.full((B, stride), -7, dtype=torch.int32, device=DEV),
        unique=torch.full((nu,), -7, dtype=torch.int32, device=DEV), sizes={}, timing=None,
        row_bytes=R)


def same(ref, got):
    rows, nu = ref.sizes["packed_rows"], ref.sizes["unique_nodes"]
    for k in ("packed_rows", "unique_nodes", "unique_packed", "total_nodes"):
        assert got.sizes[k] == ref.sizes[k], k
    assert np.array_equal(got.packed_ptr_host, ref.packed_ptr_host)
    assert torch.equal(got.packed_ptr, ref.packed_ptr)
    assert torch.equal(got.packed_ids[:rows], ref.packed_ids[:rows])
    assert torch.equal(got.unique[:nu], ref.unique[:nu])
    assert torch.equal(got.packed[:rows], ref.packed[:rows])


def run_pair(dg, w, nodes, counts, membership, clear):
    """dg_pack_group, then dg_pack_group_noalloc, on the same input; returns both."""
    X, slot = w.feats, w.cache_slot
    mem_ref = membership.clone() if membership is not None else None
    ref = dg.pack_group(X, slot, nodes, counts, with_unique=True, membership=mem_ref,
                        clear_membership=clear)
    torch.cuda.synchronize()
    got = packed_out(dg, ref, w.cfg.row_bytes)
    mem_got = membership.clone() if membership is not None else None
    got = dg.pack_group(X, slot, nodes, counts, with_unique=True, out=got, membership=mem_got,
                        clear_membership=clear, no_alloc=True)
    torch.cuda.synchronize()
    same(ref, got)
    for b in range(nodes.shape[0]):
        n = int(counts[b])
        assert torch.equal(got.loc[b, :n], ref.loc[b, :n]), b
    if clear:
        assert int(mem_got.count_nonzero()) == 0
    return ref, got


def test_noalloc_pack_matches_pack_on_calls_in_a_row(dg):
    print("[no_alloc] M1 whole group, then 8 batches, then T", flush=True)
    w = synth.make_workload("M1", device=DEV)
    mem = torch.zeros(w.cfg.n, dtype=torch.int64, device=DEV)
    sr = dg.sample_group(w.offsets, w.indices, w.seeds, list(w.cfg.fanouts), w.rng_seed,
                         membership=mem, direct=True)
    counts = sr.node_count.copy()
    need = dg._L.dg_pack_workspace_bytes(w.cfg.n, w.cfg.B, int(counts.sum()))
    assert need <= dg._L.dg_pack_noalloc_scratch_bytes(), need
    # 1: the whole M1 group, membership handed over and cleared
    run_pair(dg, w, sr.nodes, counts, mem, clear=True)
    # 2: a smaller input on the same scratch: 8 of the 32 batches, no mask given
    #    (the call builds its own mask in the scratch, which holds the last
    #    call's contents)
    run_pair(dg, w, sr.nodes[:8].contiguous(), counts[:8], None, clear=False)
    # 3: smaller still, another graph: workload T, with and without its mask
    t = synth.make_workload("T", device=DEV)
    mt = torch.zeros(t.cfg.n, dtype=torch.int64, device=DEV)
    st = dg.sample_group(t.offsets, t.indices, t.seeds, list(t.cfg.fanouts), t.rng_seed,
                         membership=mt)
    ct = st.node_count.copy()
    run_pair(dg, t, st.nodes, ct, None, clear=False)
    run_pair(dg, t, st.nodes, ct, mt, clear=False)


def test_noalloc_pack_rejects_sizes_beyond_its_scratch(dg):
    L = dg._L
    cap = L.dg_pack_noalloc_scratch_bytes()
    N = 1 << 30  # its workspace is far above the fixed scratch
    assert L.dg_pack_workspace_bytes(N, 1, 1) > cap
    fake = ctypes.c_void_p(256)  # never dereferenced: the call stops before any work
    counts = np.ones(1, dtype=np.int64)
    ptr_host = np.zeros(2, dtype=np.int64)
    sz = dg._lib.Sizes()
    rc = L.dg_pack_group_noalloc(fake, N, 16, fake, 1, fake, 1,
                                 counts.ctypes.data_as(dg._lib.I64P), 1, fake, fake, fake,
                                 ptr_host.ctypes.data_as(dg._lib.I64P), fake, None, 0, None,
                                 None, None, 0, None, 0, None, ctypes.byref(sz))
    assert rc == dg._lib.DG_EWORKSPACE
    assert b"scratch" in L.dg_last_error()
    # and the rows stream, which needs a second stream, is refused
    rc = L.dg_pack_group_noalloc(fake, 16, 16, fake, 1, fake, 1,
                                 counts.ctypes.data_as(dg._lib.I64P), 1, fake, fake, fake,
                                 ptr_host.ctypes.data_as(dg._lib.I64P), fake, None, 0, None,
                                 None, None, 0, None, dg._lib.DG_PACK_ROWS_STREAM, None,
                                 ctypes.byref(sz))
    assert rc == dg._lib.DG_EINVAL
