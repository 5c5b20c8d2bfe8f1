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


@pytest.mark.parametrize("name", ["T", "M1"])
@pytest.mark.parametrize("ranking", ["in_degree", "frequency"])
def test_cache_filled_by_the_packing_gather(dg, orc, name, ranking):
    """The cache taken as one more mini-batch of batched packing (§5.2): one
    gather launch writes the packed chunks and the cache table.  The cache table
    equals X[cache_nodes] byte for byte (empty slots left as they were), the
    packed chunks equal those of packing without it, and every batch assembled
    from this cache equals the oracle's assembly."""
    w = synth.make_workload(name, device=DEV) if name != "T" else synth.make_workload("T")
    X = w.feats.to(DEV)
    sr, mem = sampled(dg, w)
    if ranking == "in_degree":
        slot, nodes = w.cache_slot.to(DEV), w.cache_nodes.to(DEV).to(torch.int32)
    else:  # more slots than accessed nodes: the last ones stay empty (-1)
        C = int((mem != 0).sum()) + 37
        slot, nodes, cached = dg.cache_by_frequency(mem, w.cfg.B, C)
        assert cached == C - 37
    R = w.cfg.row_bytes
    C = nodes.numel()
    plain = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True)
    table = torch.full((C, R), 0xCD, dtype=torch.uint8, device=DEV)
    filled = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True,
                           cache_nodes=nodes, cache_table=table)
    torch.cuda.synchronize()
    rows = plain.sizes["packed_rows"]
    assert filled.sizes == plain.sizes
    assert torch.equal(filled.packed[:rows], plain.packed[:rows])
    full = nodes >= 0
    ref = X.index_select(0, nodes[full].long()).view(torch.uint8).reshape(-1, R)
    assert torch.equal(table[full], ref)
    assert bool((table[~full] == 0xCD).all())
    # assembly from the filled cache equals the oracle's
    Xh = w.feats.cpu().numpy()
    lists = [sr.batch_nodes(b).cpu().numpy() for b in range(w.cfg.B)]
    refp = orc.pack_group(Xh, slot.cpu().numpy(), lists)
    cache_h = table.cpu().numpy()
    for b in (0, w.cfg.B - 1):
        lo, hi = refp["packed_ptr"][b], refp["packed_ptr"][b + 1]
        y_ref = orc.assemble_batch(cache_h, refp["packed"][lo:hi], refp["loc"][b], R)
        n = len(lists[b])
        y = dg.assemble_batch(table, filled.chunk(b), filled.loc[b, :n], R)
        assert np.array_equal(y.cpu().numpy(), y_ref), b
        assert np.array_equal(y_ref, Xh.view(np.uint8).reshape(w.cfg.n, -1)[lists[b]]), b


def test_cache_fill_reports_a_bad_cache_node(dg):
    w = synth.make_workload("T")
    X = w.feats.to(DEV)
    sr, mem = sampled(dg, w)
    nodes = w.cache_nodes.to(DEV).to(torch.int32).clone()
    nodes[3] = w.cfg.n + 5
    table = torch.zeros((nodes.numel(), w.cfg.row_bytes), dtype=torch.uint8, device=DEV)
    with pytest.raises(dg.DGError) as e:
        dg.pack_group(X, w.cache_slot.to(DEV), sr.nodes, sr.node_count, cache_nodes=nodes,
                      cache_table=table)
    assert e.value.status == -1
    assert int(table[3].sum()) == 0  # its row is left as it was


@pytest.mark.parametrize("dtype,dim", [(torch.uint8, 3), (torch.float16, 5), (torch.float32, 16),
                                       (torch.float16, 768), (torch.float32, 1024)])
def test_cache_fill_every_row_shape(dg, dtype, dim):
    """The cache fill on each launch shape of the row copy (16-byte vectors and
    the narrower words of odd row sizes)."""
    n = 3000
    off, idx = synth.uniform_graph(n, 1, 12, seed=dim)
    off, idx = torch.from_numpy(off).to(DEV), torch.from_numpy(idx).to(DEV)
    gen = torch.Generator().manual_seed(dim)
    seeds = torch.stack([torch.randperm(n, generator=gen)[:40] for _ in range(3)]).to(torch.int32)
    X = torch.randint(0, 120, (n, dim), generator=gen).to(dtype).to(DEV)
    nodes = torch.randperm(n, generator=gen)[:300].to(torch.int32).to(DEV)
    nodes[7] = -1  # an empty slot
    slot = torch.full((n,), -1, dtype=torch.int32, device=DEV)
    keep = nodes >= 0
    slot[nodes[keep].long()] = torch.arange(300, dtype=torch.int32, device=DEV)[keep]
    sr = dg.sample_group(off, idx, seeds.to(DEV), [4, 3], 5)
    R = X[0].numel() * X.element_size()
    table = torch.full((300, R), 0x5A, dtype=torch.uint8, device=DEV)
    pr = dg.pack_group(X, slot, sr.nodes, sr.node_count, cache_nodes=nodes, cache_table=table)
    torch.cuda.synchronize()
    ref = X.index_select(0, nodes[keep].long()).contiguous().view(torch.uint8).reshape(-1, R)
    assert torch.equal(table[keep], ref)
    assert bool((table[7] == 0x5A).all())
    for b in range(3):
        n_b = int(sr.hop_ptr[b, -1])
        y = dg.assemble_batch(table, pr.chunk(b), pr.loc[b, :n_b], R)
        want = X.index_select(0, sr.batch_nodes(b).long()).contiguous().view(torch.uint8)
        assert torch.equal(y, want.reshape(n_b, R)), b
