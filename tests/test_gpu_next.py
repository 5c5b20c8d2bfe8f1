"""The rows built after the hot path: individual packing (the paper's naive
scheme, one gather per mini-batch) and the access-frequency cache, each
bit-exact against the oracle."""
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


def sampled(dg, w, dev=DEV):
    mem = torch.empty(w.cfg.n, dtype=torch.int64, device=dev)
    sr = dg.sample_group(w.offsets.to(dev), w.indices.to(dev), w.seeds.to(dev),
                         list(w.cfg.fanouts), w.rng_seed, membership=mem)
    return sr, mem


@pytest.mark.parametrize("name", ["T", "M1"])
def test_cache_by_frequency_matches_oracle(dg, orc, name):
    w = synth.make_workload(name, device=DEV) if name != "T" else synth.make_workload("T")
    sr, mem = sampled(dg, w)
    lists = [sr.batch_nodes(b).cpu().numpy() for b in range(w.cfg.B)]
    for pct in (0, 1, 10, 50, 100):
        C = w.cfg.n * pct // 100
        slot, nodes, cached = dg.cache_by_frequency(mem, w.cfg.B, C)
        r_slot, r_nodes, r_cached = orc.cache_by_frequency(w.cfg.n, lists, C)
        assert cached == r_cached, pct
        assert np.array_equal(slot.cpu().numpy(), r_slot), pct
        assert np.array_equal(nodes.cpu().numpy(), r_nodes), pct


def test_frequency_cache_minimises_packed_rows(dg):
    """For the same cache size, ranking by access frequency packs no more rows
    than ranking by in-degree (the placement claim of §3)."""
    w = synth.make_workload("M1", device=DEV)
    sr, mem = sampled(dg, w)
    C = w.cache_nodes.numel()
    slot_f, nodes_f, cached = dg.cache_by_frequency(mem, w.cfg.B, C)
    X = w.feats
    pf = dg.pack_group(X, slot_f, sr.nodes, sr.node_count, membership=mem)
    pd = dg.pack_group(X, w.cache_slot, sr.nodes, sr.node_count, membership=mem)
    assert pf.sizes["packed_rows"] <= pd.sizes["packed_rows"]
    # the frequency cache table filled by the row gather assembles every batch exactly
    cache = dg.gather_rows(X, nodes_f[:cached])
    for b in (0, w.cfg.B - 1):
        n = int(sr.hop_ptr[b, -1])
        y = dg.assemble_batch(cache, pf.chunk(b), pf.loc[b, :n], w.cfg.row_bytes)
        ref = X.index_select(0, sr.batch_nodes(b).long()).view(torch.uint8).reshape(n, -1)
        assert torch.equal(y, ref)


@pytest.mark.parametrize("name", ["T", "M1"])
def test_individual_packing_equals_batched(dg, orc, name):
    w = synth.make_workload(name, device=DEV) if name != "T" else synth.make_workload("T")
    sr, mem = sampled(dg, w)
    X, slot = w.feats.to(DEV), w.cache_slot.to(DEV)
    batched = dg.pack_group(X, slot, sr.nodes, sr.node_count, membership=mem)
    tables = dg.pack_group(X, slot, sr.nodes, sr.node_count, membership=mem, tables_only=True)
    rows = batched.sizes["packed_rows"]
    assert tables.sizes["packed_rows"] == rows
    assert torch.equal(tables.packed_ids[:rows], batched.packed_ids[:rows])
    indiv = torch.empty_like(batched.packed)
    dg.pack_individual(X, tables.packed_ids, tables.packed_ptr_host, indiv)
    torch.cuda.synchronize()
    assert torch.equal(indiv[:rows], batched.packed[:rows])
    if name == "T":  # and the oracle's own copies
        ref = orc.pack_group(w.feats.numpy(), w.cache_slot.numpy(),
                             [sr.batch_nodes(b).cpu().numpy() for b in range(w.cfg.B)])
        assert np.array_equal(indiv[:rows].cpu().numpy(), ref["packed"])


@pytest.mark.parametrize("dtype,dim", [(torch.float32, 16), (torch.float16, 3), (torch.uint8, 7),
                                       (torch.float32, 385)])
def test_gather_rows_any_row_size(dg, dtype, dim):
    gen = torch.Generator().manual_seed(dim)
    X = torch.randint(0, 250, (1000, dim), generator=gen).to(dtype).to(DEV)
    ids = torch.randint(0, 1000, (777,), generator=gen, dtype=torch.int32).to(DEV)
    y = dg.gather_rows(X, ids)
    torch.cuda.synchronize()
    ref = X.index_select(0, ids.long()).contiguous().view(torch.uint8).reshape(777, -1)
    assert torch.equal(y, ref)


def test_gather_rows_bad_id_flags_and_zeroes(dg):
    X = torch.ones((10, 16), dtype=torch.float32, device=DEV)
    ids = torch.tensor([1, 12, -3, 4], dtype=torch.int32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    y = dg.gather_rows(X, ids, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    assert int(y[1].sum()) == 0 and int(y[2].sum()) == 0 and int(y[0].sum()) > 0


@pytest.mark.parametrize("dim", [16, 128, 384, 512, 1024])
def test_gather_rows_bad_ids_every_row_shape(dg, dim):
    """Each launch shape of the 16-byte row gather (fp32 rows of 64 B to 4 KiB),
    over several lane groups and a ragged tail, with ids outside [0, N) at the
    first and last positions and at the int32 limits: those rows are zeroed and
    flagged, every other row is X[id]."""
    gen = torch.Generator().manual_seed(dim)
    N, n = 500, 1003
    X = torch.randn((N, dim), generator=gen).to(DEV)
    ids = torch.randint(0, N, (n,), generator=gen, dtype=torch.int32)
    bad = torch.zeros(n, dtype=torch.bool)
    for p, v in [(0, -1), (9, N), (10, 2**31 - 1), (11, -2**31), (n - 1, N + 7)]:
        ids[p] = v
        bad[p] = True
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    y = dg.gather_rows(X, ids.to(DEV), status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    got = y.cpu()
    ref = X.cpu().index_select(0, ids.clamp(0, N - 1).long()).view(torch.uint8).reshape(n, -1)
    assert int(got[bad].to(torch.int64).sum()) == 0
    assert torch.equal(got[~bad], ref[~bad])


def random_perms(k, B, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.stack([torch.randperm(B, generator=g) for _ in range(k)]).to(torch.int32)


@pytest.mark.parametrize("name,k", [("T", 1), ("T", 4), ("M1", 3)])
def test_minhash_order_matches_oracle(dg, orc, name, k):
    w = synth.make_workload(name, device=DEV) if name != "T" else synth.make_workload("T")
    sr, mem = sampled(dg, w)
    lists = [sr.batch_nodes(b).cpu().numpy() for b in range(w.cfg.B)]
    # disk-cache entries: the non-cached accessed nodes plus a few never accessed
    accessed = (mem != 0).nonzero().squeeze(1)
    slot = w.cache_slot.to(DEV)
    entries = accessed[slot[accessed] < 0]
    extra = ((mem == 0).nonzero().squeeze(1))[:100]
    entries = torch.cat([entries, extra]).to(torch.int32)
    g = torch.Generator().manual_seed(k)
    entries = entries[torch.randperm(entries.numel(), generator=g).to(DEV)].contiguous()
    perms = random_perms(k, w.cfg.B, 11 * k)
    order, sig = dg.minhash_order(mem, w.cfg.B, entries, perms.to(DEV))
    r_order, r_sig = orc.minhash_order(w.cfg.n, lists, entries.cpu().numpy(), perms.numpy())
    assert np.array_equal(sig.cpu().numpy(), r_sig)
    assert np.array_equal(order.cpu().numpy(), r_order)


def test_minhash_rejects_bad_hash_values(dg):
    mem = torch.zeros(10, dtype=torch.int64, device=DEV)
    mem[3] = 1
    entries = torch.tensor([3, 4], dtype=torch.int32, device=DEV)
    perms = torch.tensor([[0, 5]], dtype=torch.int32, device=DEV)
    with pytest.raises(dg.DGError):
        dg.minhash_order(mem, 2, entries, perms)
