"""The pipelined loop bench.py times, checked for correctness under real
concurrency.  Sampling and packing run on one stream, the row copy and the
assembly on a second one, with two packing output sets and two packing
workspaces; each packing call waits for the assembly that last read its set;
the clearing flags and the member-lines map carry state from step to step;
sampling writes the cached nodes' address-table entries into the step's
packing set, which packing completes.
Every step takes a different seed group, so an output read or written by the
wrong step would show up as a wrong row.  Each step assembles into buffers of
its own, and all are checked against a library gather (torch.index_select) at
the end.  The loop runs on M1 in both call forms, and on L100 at full size in
the benchmark's exact form (one call per step, the assembly issued from a
host thread of its own)."""
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


@pytest.mark.parametrize("fused", [False, True])
def test_pipelined_steps_are_each_correct(dg, fused):
    """fused: each step samples and packs in one dg_sample_pack_group call,
    with a packing workspace per output set."""
    w = synth.make_workload("M1", device=DEV)
    cfg = w.cfg
    fan = list(cfg.fanouts)
    B, R, steps = cfg.B, cfg.row_bytes, 6
    groups = [synth.seed_batches(cfg.n, B, cfg.S, cfg.seed + 100 + k, DEV, offsets=w.offsets)
              for k in range(steps)]
    node_cap, edge_cap = dg.sample_bounds(cfg.n, w.num_edges, cfg.S, fan)
    flags = dg.sample_flags(direct=True)
    ws_s = torch.empty(dg._L.dg_sample_workspace_bytes(cfg.n, B, node_cap, edge_cap, flags),
                       dtype=torch.uint8, device=DEV)
    ws_p = [torch.empty(dg._L.dg_sample_pack_workspace_bytes(cfg.n, B, node_cap) if fused
                        else dg._L.dg_pack_workspace_bytes(cfg.n, B, B * node_cap),
                        dtype=torch.uint8, device=DEV) for _ in range(2)]
    mem = torch.empty(cfg.n, dtype=torch.int64, device=DEV)
    lines = torch.empty(dg.member_lines_bytes(cfg.n), dtype=torch.uint8, device=DEV)
    # output capacity fixed up front (the largest group) so every step reuses it
    sizes = []
    for g in groups:
        sr = dg.sample_group(w.offsets, w.indices, g, fan, w.rng_seed, direct=True)
        pr = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count)
        sizes.append((int(sr.node_count.max()), pr.sizes["packed_rows"]))
    nmax = max(s[0] for s in sizes)
    rows_max = max(s[1] for s in sizes)
    pr2 = []
    for _ in range(2):
        pr_ = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count)
        pr_.packed = torch.empty((rows_max, R), dtype=torch.uint8, device=DEV)
        pr_.packed_ids = torch.empty(rows_max, dtype=torch.int32, device=DEV)
        pr2.append(pr_)
    kept = [[torch.empty((nmax, R), dtype=torch.uint8, device=DEV) for _ in range(B)]
            for _ in range(steps)]
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    s_asm = torch.cuda.Stream(device=DEV)
    asm_done = [torch.cuda.Event(), torch.cuda.Event()]
    pack_done = torch.cuda.Event()
    for e in asm_done:
        e.record(s_asm)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    results = []
    clear = False
    for k in range(steps):
        slot = k & 1
        print(f"[pipeline] step {k}", flush=True)
        # sampling writes the cached nodes' address-table entries into this
        # step's packing set, so it waits for the assembly that last read it
        stream.wait_event(asm_done[slot])
        if fused:
            sr, pr = dg.sample_pack_group(w.offsets, w.indices, groups[k], fan, w.rng_seed,
                                          w.feats, w.cache_slot, node_cap=node_cap,
                                          edge_cap=edge_cap, pack_out=pr2[slot],
                                          workspace=ws_s, pack_workspace=ws_p[slot],
                                          stream=stream, rows_stream=s_asm, membership=mem,
                                          direct=True, exit_clear=True, entry_clear=clear)
            counts = sr.node_count.copy()
            nodes = sr.nodes.clone()
        else:
            sr = dg.sample_group(w.offsets, w.indices, groups[k], fan, w.rng_seed,
                                 membership=mem, workspace=ws_s, direct=True, exit_clear=True,
                                 entry_clear=clear, member_lines=lines, stream=stream,
                                 cache_slot=w.cache_slot, loc=pr2[slot].loc, node_cap=node_cap,
                                 edge_cap=edge_cap)
            counts = sr.node_count.copy()
            nodes = sr.nodes.clone()  # the next step's sampling overwrites sr.nodes
            pr = dg.pack_group(w.feats, w.cache_slot, sr.nodes, counts, out=pr2[slot],
                               workspace=ws_p[slot], membership=mem, clear_membership=True,
                               member_lines=lines, stream=stream, rows_stream=s_asm,
                               loc_pending=True)
        clear = True
        pack_done.record(stream)
        s_asm.wait_event(pack_done)
        # one output buffer per batch and step, so that every step's rows stay
        # for the check (the bench uses eight buffers in turn instead)
        dg.assemble_batches(w.cache, pr, counts, kept[k], status=status, stream=s_asm)
        asm_done[slot].record(s_asm)
        results.append((nodes, counts))
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert int(mem.count_nonzero()) == 0
    for k, (nodes, counts) in enumerate(results):
        for b in range(B):
            n = int(counts[b])
            ref = w.feats.index_select(0, nodes[b, :n].long()).view(torch.uint8).reshape(n, R)
            assert torch.equal(kept[k][b][:n], ref), (k, b)


@pytest.mark.big
@pytest.mark.timeout(900)
def test_pipelined_steps_full_size_L100(dg):
    """The benchmark's own loop at full size (L100): one dg_sample_pack_group
    call per step on the main thread with the row copy queued on the assembly
    stream, two packing output sets and workspaces, the clearing flags, and each
    step's dg_assemble_batches issued from a host thread of its own once that
    step's packing is recorded.  Four steps, four distinct seed groups with
    their own global batch numbers; every assembled row of every step is checked
    against a library gather of the feature table."""
    import queue
    import threading

    w = synth.make_workload("L100", device=DEV)
    cfg = w.cfg
    fan, B, R, steps = list(cfg.fanouts), cfg.B, cfg.row_bytes, 4
    groups = [w.seeds] + [synth.seed_batches(cfg.n, 2 * B, cfg.S, cfg.seed, DEV,
                                             offsets=w.offsets)[B:]]
    groups += [synth.seed_batches(cfg.n, 4 * B, cfg.S, cfg.seed, DEV,
                                  offsets=w.offsets)[k * B:(k + 1) * B] for k in (2, 3)]
    node_cap, edge_cap = dg.sample_bounds(cfg.n, w.num_edges, cfg.S, fan)
    ws_s = torch.empty(dg._L.dg_sample_workspace_bytes(cfg.n, B, node_cap, edge_cap,
                                                       dg.sample_flags(direct=True)),
                       dtype=torch.uint8, device=DEV)
    ws_p = [torch.empty(dg._L.dg_sample_pack_workspace_bytes(cfg.n, B, node_cap),
                        dtype=torch.uint8, device=DEV) for _ in range(2)]
    mem = torch.empty(cfg.n, dtype=torch.int64, device=DEV)
    # output capacity for the largest group, sized by a tables-only pass
    rows_max, nmax = 0, 0
    for k, g in enumerate(groups):
        sr = dg.sample_group(w.offsets, w.indices, g, fan, w.rng_seed, batch_base=k * B,
                             direct=True, workspace=ws_s, membership=mem, node_cap=node_cap,
                             edge_cap=edge_cap)
        pr = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count, tables_only=True,
                           membership=mem)
        rows_max = max(rows_max, pr.sizes["packed_rows"])
        nmax = max(nmax, int(sr.node_count.max()))
        del pr
    sets = [dg.PackResult(packed=torch.empty((rows_max, R), dtype=torch.uint8, device=DEV),
                          packed_ids=torch.empty(rows_max, dtype=torch.int32, device=DEV),
                          packed_ptr=torch.empty(B + 1, dtype=torch.int64, device=DEV),
                          packed_ptr_host=np.zeros(B + 1, dtype=np.int64),
                          loc=torch.empty((B, node_cap), dtype=torch.int32, device=DEV),
                          unique=None, sizes={}, timing=None, row_bytes=R) for _ in range(2)]
    kept = [[torch.empty((nmax, R), dtype=torch.uint8, device=DEV) for _ in range(B)]
            for _ in range(steps)]
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    s_asm = torch.cuda.Stream(device=DEV)
    asm_done = [torch.cuda.Event(), torch.cuda.Event()]
    pack_done = [torch.cuda.Event(), torch.cuda.Event()]
    for e in asm_done + pack_done:
        e.record(s_asm)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    free = [threading.Event(), threading.Event()]
    for f in free:
        f.set()
    q, errors = queue.Queue(), []

    def assembler():
        while True:
            item = q.get()
            if item is None:
                return
            k, slot, pr, counts = item
            try:
                s_asm.wait_event(pack_done[slot])
                dg.assemble_batches(w.cache, pr, counts, kept[k], status=status, stream=s_asm)
                asm_done[slot].record(s_asm)
            except Exception as e:  # reported by the main thread
                errors.append(e)
            finally:
                free[slot].set()

    t = threading.Thread(target=assembler, daemon=True)
    t.start()
    results = []
    for k in range(steps):
        slot = k & 1
        print(f"[pipeline L100] step {k}", flush=True)
        free[slot].wait()
        free[slot].clear()
        stream.wait_event(asm_done[slot])
        sr, pr = dg.sample_pack_group(w.offsets, w.indices, groups[k], fan, w.rng_seed,
                                      w.feats, w.cache_slot, batch_base=k * B,
                                      node_cap=node_cap, edge_cap=edge_cap, pack_out=sets[slot],
                                      workspace=ws_s, pack_workspace=ws_p[slot], stream=stream,
                                      rows_stream=s_asm, membership=mem, direct=True,
                                      exit_clear=True, entry_clear=k > 0)
        counts = sr.node_count.copy()
        results.append((sr.nodes.clone(), counts))  # the next step overwrites sr.nodes
        pack_done[slot].record(stream)
        q.put((k, slot, pr, counts))
    q.put(None)
    t.join(timeout=300)
    assert not t.is_alive() and not errors, errors
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert int(mem.count_nonzero()) == 0
    for k, (nodes, counts) in enumerate(results):
        for b in range(B):
            n = int(counts[b])
            ref = w.feats.index_select(0, nodes[b, :n].long()).view(torch.uint8).reshape(n, R)
            assert torch.equal(kept[k][b][:n], ref), (k, b)


def test_two_host_threads_at_once(dg):
    """The library keeps host state per thread only (error text, side streams,
    events, staging): two host threads, each with its own stream, workspaces
    and membership buffer, sample and pack different groups at the same time
    (ctypes releases the interpreter lock during each call), and every result
    equals that of the same group run alone."""
    import threading

    from test_gpu_clear import same_pack, same_sample
    w = synth.make_workload("M1", device=DEV)
    cfg = w.cfg
    fan, B = list(cfg.fanouts), cfg.B
    groups = [synth.seed_batches(cfg.n, B, cfg.S, cfg.seed + 300 + k, DEV, offsets=w.offsets)
              for k in range(4)]
    refs = []
    for k, g in enumerate(groups):
        sr = dg.sample_group(w.offsets, w.indices, g, fan, w.rng_seed, batch_base=k * B,
                             direct=True)
        pr = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count, with_unique=True)
        refs.append((sr, pr))
    torch.cuda.synchronize()
    results, errors = [None] * len(groups), []

    def worker(ks):
        try:
            s = torch.cuda.Stream(device=DEV)
            with torch.cuda.stream(s):
                for k in ks:
                    mem = torch.empty(cfg.n, dtype=torch.int64, device=DEV)
                    sr = dg.sample_group(w.offsets, w.indices, groups[k], fan, w.rng_seed,
                                         batch_base=k * B, membership=mem, direct=True,
                                         stream=s)
                    pr = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count,
                                       with_unique=True, membership=mem, stream=s)
                    results[k] = (sr, pr)
            s.synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(ks,)) for ks in ([0, 2], [1, 3])]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=100)
    assert not any(t.is_alive() for t in threads)
    assert not errors, errors
    for k, (sr, pr) in enumerate(results):
        same_sample(sr, refs[k][0])
        same_pack(pr, refs[k][1], sr.node_count)
