"""Error paths of the device library, forced from the host with bad inputs or
small capacities: every kernel still runs to completion and stays inside its
buffers; the call reports the problem."""
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


@pytest.fixture(scope="module")
def tiny():
    w = synth.make_workload("T")
    return w


@pytest.mark.parametrize("direct", [False, True])
def test_duplicate_seed_rejected(dg, tiny, direct):
    seeds = tiny.seeds.clone()
    seeds[1, 5] = seeds[1, 9]
    with pytest.raises(dg.DGError) as e:
        dg.sample_group(tiny.offsets.to(DEV), tiny.indices.to(DEV), seeds.to(DEV), [5, 5], 1, direct=direct)
    assert e.value.status == -1 and "twice" in str(e.value)


@pytest.mark.parametrize("direct", [False, True])
def test_seed_out_of_range_rejected(dg, tiny, direct):
    seeds = tiny.seeds.clone()
    seeds[0, 0] = tiny.cfg.n + 3
    with pytest.raises(dg.DGError) as e:
        dg.sample_group(tiny.offsets.to(DEV), tiny.indices.to(DEV), seeds.to(DEV), [5, 5], 1, direct=direct)
    assert e.value.status == -1 and "outside" in str(e.value)


@pytest.mark.parametrize("direct", [False, True])
def test_bad_neighbour_id_rejected(dg, tiny, direct):
    idx = tiny.indices.clone()
    idx[::7] = -5
    with pytest.raises(dg.DGError) as e:
        dg.sample_group(tiny.offsets.to(DEV), idx.to(DEV), tiny.seeds.to(DEV), [5, 5], 1,
                        direct=direct)
    assert e.value.status == -1 and "neighbour" in str(e.value)


@pytest.mark.parametrize("direct", [False, True])
def test_bad_offsets_rejected(dg, tiny, direct):
    off = tiny.offsets.clone()
    off[100:200] = 10 ** 9  # beyond num_edges
    seeds = torch.arange(100, 164, dtype=torch.int32).reshape(1, 64)
    with pytest.raises(dg.DGError) as e:
        dg.sample_group(off.to(DEV), tiny.indices.to(DEV), seeds.to(DEV), [5, 5], 1, direct=direct)
    assert e.value.status == -1 and "CSR" in str(e.value)


def test_sample_capacity_reported(dg, tiny):
    off, idx, seeds = tiny.offsets.to(DEV), tiny.indices.to(DEV), tiny.seeds.to(DEV)
    full = dg.sample_group(off, idx, seeds, [5, 5], 1)
    need_n = full.sizes["max_batch_nodes"]
    need_e = full.sizes["max_batch_edges"]
    # node capacity one short: hop 2 overflows; outputs never written past the cap
    B = seeds.shape[0]
    guard = 4096
    nodes = torch.full((B * (need_n - 1) + guard,), 7777, dtype=torch.int32, device=DEV)
    res = dg.SampleResult(nodes=nodes[:B * (need_n - 1)].view(B, need_n - 1),
                          hop_ptr=np.zeros((B, 4), dtype=np.int64),
                          edge_src=torch.empty((B, need_e), dtype=torch.int32, device=DEV),
                          edge_dst=torch.empty((B, need_e), dtype=torch.int32, device=DEV),
                          edge_ptr=np.zeros((B, 3), dtype=np.int64), sizes={}, timing=None)
    with pytest.raises(dg.DGError) as e:
        dg.sample_group(off, idx, seeds, [5, 5], 1, out=res)
    assert e.value.status == -2
    assert res.sizes["max_batch_nodes"] >= need_n - 1 + 1 or res.sizes["exact"] == 0
    assert bool((nodes[B * (need_n - 1):] == 7777).all())
    # edge capacity one short (both relabelling modes)
    for direct in (False, True):
        es = torch.full((B * (need_e - 1) + guard,), 7777, dtype=torch.int32, device=DEV)
        ed = torch.full((B * (need_e - 1) + guard,), 7777, dtype=torch.int32, device=DEV)
        res2 = dg.SampleResult(nodes=torch.empty((B, need_n), dtype=torch.int32, device=DEV),
                               hop_ptr=np.zeros((B, 4), dtype=np.int64),
                               edge_src=es[:B * (need_e - 1)].view(B, need_e - 1),
                               edge_dst=ed[:B * (need_e - 1)].view(B, need_e - 1),
                               edge_ptr=np.zeros((B, 3), dtype=np.int64), sizes={}, timing=None)
        with pytest.raises(dg.DGError) as e:
            dg.sample_group(off, idx, seeds, [5, 5], 1, out=res2, direct=direct)
        assert e.value.status == -2 and res2.sizes["max_batch_edges"] == need_e
        assert bool((es[B * (need_e - 1):] == 7777).all())
        assert bool((ed[B * (need_e - 1):] == 7777).all())


def test_pack_duplicate_and_range_rejected(dg, tiny):
    X = tiny.feats.to(DEV)
    slot = tiny.cache_slot.to(DEV)
    nodes = torch.tensor([[1, 2, 3, 2], [4, 5, 6, 7]], dtype=torch.int32, device=DEV)
    with pytest.raises(dg.DGError) as e:
        dg.pack_group(X, slot, nodes, [4, 4])
    assert e.value.status == -1 and "twice" in str(e.value)
    nodes = torch.tensor([[1, 2, 3, 10 ** 6]], dtype=torch.int32, device=DEV)
    with pytest.raises(dg.DGError) as e:
        dg.pack_group(X, slot, nodes, [4])
    assert e.value.status == -1 and "outside" in str(e.value)
    bad = slot.clone()
    bad[3] = -7
    nodes = torch.tensor([[1, 2, 3]], dtype=torch.int32, device=DEV)
    with pytest.raises(dg.DGError) as e:
        dg.pack_group(X, bad, nodes, [3])
    assert e.value.status == -1 and "cache_slot" in str(e.value)


def test_pack_capacity_reported(dg, tiny):
    X = tiny.feats.to(DEV)
    slot = torch.full((tiny.cfg.n,), -1, dtype=torch.int32, device=DEV)
    nodes = torch.tensor([[1, 2, 3, 4], [3, 4, 5, 6]], dtype=torch.int32, device=DEV)
    full = dg.pack_group(X, slot, nodes, [4, 4], with_unique=True)
    assert full.sizes["packed_rows"] == 8 and full.sizes["unique_nodes"] == 6
    R = tiny.cfg.row_bytes
    guard = torch.full((8 * R,), 0xAB, dtype=torch.uint8, device=DEV)
    small = dg.PackResult(packed=guard[:7 * R].view(7, R),
                          packed_ids=torch.empty(7, dtype=torch.int32, device=DEV),
                          packed_ptr=torch.empty(3, dtype=torch.int64, device=DEV),
                          packed_ptr_host=np.zeros(3, dtype=np.int64),
                          loc=torch.empty((2, 4), dtype=torch.int32, device=DEV),
                          unique=None, sizes={}, timing=None, row_bytes=R)
    with pytest.raises(dg.DGError) as e:
        dg.pack_group(X, slot, nodes, [4, 4], out=small)
    assert e.value.status == -2 and small.sizes["packed_rows"] == 8
    assert bool((guard == 0xAB).all())  # nothing written anywhere


def test_assemble_bad_address_flags_and_zeroes(dg):
    R = 64
    cache = torch.arange(4 * R, dtype=torch.int32, device=DEV).to(torch.uint8).view(4, R)
    packed = torch.full((3, R), 9, dtype=torch.uint8, device=DEV)
    loc = torch.tensor([-1, 0, 5, -9, 2], dtype=torch.int32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = dg.assemble_batch(cache, packed, loc, R, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    assert torch.equal(out[0], cache[0]) and torch.equal(out[1], packed[0])
    assert torch.equal(out[4], packed[2])
    assert int(out[2].sum()) == 0 and int(out[3].sum()) == 0


def test_assemble_batches_bad_address_flags(dg):
    """The group call checks addresses like the per-batch call: an entry outside
    its table is flagged and its row zeroed; the other batches are untouched."""
    R = 64
    cache = torch.arange(4 * R, dtype=torch.int32, device=DEV).to(torch.uint8).view(4, R)
    packed = torch.full((5, R), 9, dtype=torch.uint8, device=DEV)
    packed[3:] = 7
    loc = torch.tensor([[-1, 0, 7], [1, -2, 0]], dtype=torch.int32, device=DEV)  # 7: beyond chunk 0
    pr = dg.PackResult(packed=packed, packed_ids=torch.zeros(5, dtype=torch.int32, device=DEV),
                       packed_ptr=torch.tensor([0, 3, 5], dtype=torch.int64, device=DEV),
                       packed_ptr_host=np.array([0, 3, 5], dtype=np.int64), loc=loc,
                       unique=None, sizes={}, timing=None, row_bytes=R)
    outs = [torch.full((3, R), 0xCD, dtype=torch.uint8, device=DEV) for _ in range(2)]
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    dg.assemble_batches(cache, pr, [3, 3], outs, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    assert torch.equal(outs[0][0], cache[0]) and torch.equal(outs[0][1], packed[0])
    assert int(outs[0][2].sum()) == 0
    assert torch.equal(outs[1][0], packed[4]) and torch.equal(outs[1][1], cache[1])
    assert torch.equal(outs[1][2], packed[3])



@pytest.mark.parametrize("R", [64, 512, 1536, 2048, 4096])
def test_assemble_bad_entries_every_row_shape(dg, R):
    """Every launch shape of the 16-byte path (one to four vectors per lane,
    the last one partly used at 1536 bytes), over several lane groups and a
    ragged tail: entries outside both tables, the int32 limits among them, are
    flagged and their rows zeroed; every other row is the addressed one."""
    g = torch.Generator().manual_seed(R)
    n_cache, n_packed, n = 40, 30, 1003
    cache = torch.randint(0, 256, (n_cache, R), generator=g, dtype=torch.int32).to(torch.uint8)
    packed = torch.randint(0, 256, (n_packed, R), generator=g, dtype=torch.int32).to(torch.uint8)
    loc = torch.randint(-n_cache, n_packed, (n,), generator=g, dtype=torch.int32)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = dg.assemble_batch(cache.to(DEV), packed.to(DEV), loc.to(DEV), R, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    want = torch.where((loc < 0).unsqueeze(1), cache[(-loc - 1).clamp(min=0).long()],
                       packed[loc.clamp(min=0).long()])
    assert torch.equal(out.cpu(), want)
    for p, v in [(0, -n_cache - 1), (5, n_packed), (6, 2**31 - 1), (7, -2**31), (500, 31),
                 (n - 1, -1000)]:
        loc[p] = v
    bad = torch.zeros(n, dtype=torch.bool)
    bad[[0, 5, 6, 7, 500, n - 1]] = True
    out = dg.assemble_batch(cache.to(DEV), packed.to(DEV), loc.to(DEV), R, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 1
    got = out.cpu()
    assert int(got[bad].to(torch.int64).sum()) == 0
    assert torch.equal(got[~bad], want[~bad])


def handoff_setup(dg, tiny):
    off, idx = tiny.offsets.to(DEV), tiny.indices.to(DEV)
    seeds = tiny.seeds.to(DEV)
    ncap, ecap = dg.sample_bounds(tiny.cfg.n, tiny.num_edges, tiny.cfg.S, [5, 5])
    loc = torch.full((tiny.cfg.B, ncap), -3, dtype=torch.int32, device=DEV)
    return off, idx, seeds, ncap, ecap, loc


@pytest.mark.parametrize("direct", [False, True])
def test_handoff_bad_cache_slot_rejected_by_sampling(dg, tiny, direct):
    """A cache_slot value below -1 given to sampling for the address tables."""
    off, idx, seeds, ncap, ecap, loc = handoff_setup(dg, tiny)
    slot = tiny.cache_slot.to(DEV).clone()
    slot[::3] = -9  # reaches seeds and sampled nodes alike
    with pytest.raises(dg.DGError) as e:
        dg.sample_group(off, idx, seeds, [5, 5], 1, direct=direct, node_cap=ncap, edge_cap=ecap,
                        cache_slot=slot, loc=loc)
    assert e.value.status == -1 and "cache_slot" in str(e.value)


def test_handoff_pending_entry_of_a_cached_node_rejected(dg, tiny):
    """Packing told that loc came from sampling with another cache_slot: a
    pending entry whose node is cached now has no packed row, and is reported;
    the entries it keeps are never followed."""
    off, idx, seeds, ncap, ecap, loc = handoff_setup(dg, tiny)
    X = tiny.feats.to(DEV)
    slot = tiny.cache_slot.to(DEV)
    sr = dg.sample_group(off, idx, seeds, [5, 5], 1, node_cap=ncap, edge_cap=ecap,
                         cache_slot=slot, loc=loc)
    ref = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True)
    # a node that was not cached at sampling time becomes cached
    u = int(sr.batch_nodes(1)[3])
    assert int(slot[u]) == -1
    slot2 = slot.clone()
    slot2[u] = 0
    out = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True)  # buffers
    out.loc.copy_(loc)
    with pytest.raises(dg.DGError) as e:
        dg.pack_group(X, slot2, sr.nodes, sr.node_count, with_unique=True, out=out,
                      loc_pending=True)
    assert e.value.status == -1
    # and with the same cache_slot the completed table equals packing's own
    out.loc.copy_(loc)
    pr = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True, out=out,
                       loc_pending=True)
    for b in range(tiny.cfg.B):
        n = int(sr.hop_ptr[b, -1])
        assert torch.equal(pr.loc[b, :n], ref.loc[b, :n]), b


@pytest.mark.parametrize("direct", [False, True])
def test_sample_pack_errors_and_capacity(dg, tiny, direct):
    """dg_sample_pack_group: a bad cache slot is reported (in the fused pass and
    in packing's own passes alike); too little packed or unique room gives
    DG_ECAPACITY with the sizes needed, and writes nothing past the buffers; a
    call with room afterwards (without DG_SAMPLE_ENTRY_CLEAR) equals the
    separate calls."""
    off, idx, seeds, ncap, ecap, loc = handoff_setup(dg, tiny)
    X = tiny.feats.to(DEV)
    slot = tiny.cache_slot.to(DEV)
    bad = slot.clone()
    bad[::3] = -9
    with pytest.raises(dg.DGError) as e:
        dg.sample_pack_group(off, idx, seeds, [5, 5], 1, X, bad, node_cap=ncap, edge_cap=ecap,
                             direct=direct)
    assert e.value.status == -1 and "cache_slot" in str(e.value)
    sr = dg.sample_group(off, idx, seeds, [5, 5], 1, direct=direct, node_cap=ncap,
                         edge_cap=ecap)
    ref = dg.pack_group(X, slot, sr.nodes, sr.node_count, with_unique=True)
    rows, nu = ref.sizes["packed_rows"], ref.sizes["unique_nodes"]
    B, R = tiny.cfg.B, ref.row_bytes
    mem = torch.empty(tiny.cfg.n, dtype=torch.int64, device=DEV)
    # a guard element after each list output, which must stay untouched
    ids = torch.full((rows + 1,), -11, dtype=torch.int32, device=DEV)
    uq = torch.full((nu + 1,), -11, dtype=torch.int32, device=DEV)
    packed = torch.full((rows + 1, R), 5, dtype=torch.uint8, device=DEV)

    def out_set(n_rows, n_u):
        return dg.PackResult(packed=packed[:n_rows], packed_ids=ids[:n_rows],
                             packed_ptr=torch.empty(B + 1, dtype=torch.int64, device=DEV),
                             packed_ptr_host=np.zeros(B + 1, dtype=np.int64), loc=loc,
                             unique=uq[:n_u], sizes={}, timing=None, row_bytes=R)

    for n_rows, n_u in ((rows - 1, nu), (rows, nu - 1)):
        with pytest.raises(dg.DGError) as e:
            dg.sample_pack_group(off, idx, seeds, [5, 5], 1, X, slot, node_cap=ncap,
                                 edge_cap=ecap, pack_out=out_set(n_rows, n_u), membership=mem,
                                 direct=direct, exit_clear=True)
        assert e.value.status == -2
        assert int(ids[rows]) == -11 and int(uq[nu]) == -11
        assert int(packed[rows].to(torch.int64).sum()) == 5 * R
    sr2, pr2 = dg.sample_pack_group(off, idx, seeds, [5, 5], 1, X, slot, node_cap=ncap,
                                    edge_cap=ecap, pack_out=out_set(rows, nu), membership=mem,
                                    direct=direct, exit_clear=True)
    assert pr2.sizes["packed_rows"] == rows and pr2.sizes["unique_nodes"] == nu
    assert torch.equal(pr2.packed_ids[:rows], ref.packed_ids[:rows])
    assert torch.equal(pr2.unique[:nu], ref.unique[:nu])
    assert torch.equal(pr2.packed[:rows], ref.packed[:rows])
    for b in range(B):
        n = int(sr.hop_ptr[b, -1])
        assert torch.equal(sr2.nodes[b, :n], sr.nodes[b, :n]), b
        assert torch.equal(pr2.loc[b, :n], ref.loc[b, :n]), b
    assert int(ids[rows]) == -11 and int(uq[nu]) == -11
    assert int(mem.count_nonzero()) == 0
