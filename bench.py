"""Benchmark of the offline-sampling hot path on one MI355X.

One step = one pass of the whole path over a group of mini-batches whose
inputs are resident in HBM: group sampling (dg_sample_group) -> batched
packing (dg_pack_group) -> assembly of every mini-batch (dg_assemble_batch).

Reported value: feature bytes the method must move per step (packing: each
non-cached unique row read once + one row write per packed row; assembly: one
row read + one row write per required row) divided by the wall time of the
whole step, in GB/s.  Sampled edges/s, per-phase rates and the roofline
fraction of the fan-out gather kernel are reported beside it, with the CPU
oracle timed on a bounded sample of the same workload.

Usage: python bench.py [--steps K] [--warmup W] [--workload L100] [--gpus 1]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import queue
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
# mini-batches per assembly launch in dg_assemble_batches (when their output
# buffers are distinct)
ASM_GROUP = 8


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# The translation units of the two row kernels: each source and the headers it
# includes.
KERNEL_TU = {"fanout_gather": ("dg_gather.hip", "dg_common.h", "dg_rows.h"),
             "assemble": ("dg_assemble.hip", "dg_common.h", "dg_rows.h")}
GATHER_TU = KERNEL_TU["fanout_gather"]


def kernel_source_digest(kernel: str = "fanout_gather") -> str:
    """Digest of the sources a roofline kernel is built from (ties committed
    counter readings to the code they were taken on)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2405_05231_amd", "csrc")
    for name in KERNEL_TU[kernel]:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def load_traffic(workload: str, kernel: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_digest") != kernel_source_digest(kernel):
        return None
    return t.get("bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="L100")
    ap.add_argument("--cache-pct", type=int, default=None)
    ap.add_argument("--cpu-batches", type=int, default=0,
                    help="mini-batches in the CPU-oracle sample (0 = the whole group)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sample-timing", action="store_true",
                    help="time the sampling call's phases (draw, compaction, relabelling) with "
                         "the library's HIP events in both regions and report their medians")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the row-copy ceiling measured after the timed regions")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="time the serial region only (value = the serial rate)")
    ap.add_argument("--timed-pack", action="store_true",
                    help="request per-phase timing from every packing call (its phases then "
                         "run one after the other, so a kernel trace sees the fan-out gather "
                         "alone in every call)")
    ap.add_argument("--no-member-lines", action="store_true",
                    help="packing reads every membership word instead of only the lines "
                         "sampling marked as holding a member (comparison)")
    ap.add_argument("--rows-inline", action="store_true",
                    help="pipelined region: keep packing's row copy inside the packing call "
                         "instead of queueing it on the assembly stream (comparison)")
    ap.add_argument("--no-loc-handoff", action="store_true",
                    help="packing builds every address-table entry itself, instead of "
                         "completing the ones sampling wrote for cached nodes (comparison)")
    ap.add_argument("--two-calls", action="store_true",
                    help="sample with dg_sample_group and pack with dg_pack_group, instead of "
                         "one dg_sample_pack_group call whose last compaction pass also does "
                         "packing's pass (comparison)")
    ap.add_argument("--sets", type=int, default=2,
                    help="packing output sets (and workspaces) used in turn: step k waits for "
                         "the assembly of step k - sets before it writes into its set")
    ap.add_argument("--asm-inline", action="store_true",
                    help="pipelined region: issue each step's assembly from the main thread "
                         "instead of a host thread of its own (comparison)")
    ap.add_argument("--fill-masks", action="store_true",
                    help="clear the membership mask and the sampler's state with full fills "
                         "in every sampling call, instead of the clearing flags (comparison)")
    ap.add_argument("--copy-calib", action="store_true",
                    help="also run a plain copy of known size (counter calibration)")
    ap.add_argument("--groups", type=int, default=16,
                    help="groups of B mini-batches for --experiment regime")
    ap.add_argument("--experiment",
                    choices=["pack_ab", "cache", "cache_fill", "layered", "minhash", "regime",
                             "ceiling"],
                    default=None,
                    help="instead of the step benchmark: batched vs individual packing "
                         "(pack_ab), access-frequency vs in-degree cache (cache), the cache "
                         "filled by the packing gather vs a separate gather (cache_fill), or "
                         "layer-wise (DGL-style) vs new-node frontier sampling (layered), or "
                         "disk-cache pages touched under ID vs MinHash order (minhash), or "
                         "the node access distribution over several groups (regime), or "
                         "the rate of plain row copies on this memory system (ceiling)")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0 or args.sets < 2:
        ap.error("--steps must be at least 1, --warmup at least 0 and --sets at least 2")
    if not args.two_calls and (args.no_loc_handoff or args.no_member_lines):
        ap.error("--no-loc-handoff and --no-member-lines compare options of the two-call path: "
                 "add --two-calls")

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the hot path is measured on one GPU's "
              "share of the work; running it across several GPUs is not implemented.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2405_05231_amd as dg
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = synth.CONFIGS[args.workload]
    t0 = time.perf_counter()
    log(f"generating {cfg.name}: N={cfg.n:,} draws={cfg.draws:,} dim={cfg.dim} {cfg.dtype}")
    w = synth.make_workload(cfg, device=dev, cache_pct=args.cache_pct)
    torch.cuda.synchronize()
    log(f"workload ready in {time.perf_counter() - t0:.1f}s: E={w.num_edges:,} "
        f"cache={w.cache_nodes.numel():,} rows")
    torch.cuda.empty_cache()

    fan = list(cfg.fanouts)
    R = cfg.row_bytes
    B = cfg.B
    stream = torch.cuda.current_stream()
    if args.experiment:
        out = {"pack_ab": experiment_pack_ab, "cache": experiment_cache,
               "cache_fill": experiment_cache_fill,
               "layered": experiment_layered,
               "minhash": experiment_minhash,
               "ceiling": experiment_ceiling,
               "regime": lambda *a: experiment_regime(*a, groups=args.groups)}[args.experiment](
                   dg, w, cfg, args.steps)
        print(json.dumps(out), flush=True)
        return

    # The stream of groups.  Offline sampling (§3) samples many mini-batches
    # ahead of training: here consecutive groups of B mini-batches from one seed
    # stream (seeds drawn without replacement across the whole stream, so no
    # two groups share a seed; group g holds global mini-batches g*B .. g*B+B-1).
    # Every timed step takes a group of its own: the serial region the first
    # warmup+steps groups, the pipelined region the next ones.  Group 0 is the
    # workload's own group.
    n_region = args.warmup + args.steps
    n_groups = 2 * n_region
    # A graph with fewer seed candidates (nodes with out-neighbours) than the
    # stream needs reuses its seed groups in turn; every step still keeps its own
    # global batch numbers, so its draws differ.
    candidates = int((w.offsets[1:] > w.offsets[:-1]).sum())
    n_seed_groups = max(1, min(n_groups, candidates // (B * cfg.S)))
    seeds_all = synth.seed_batches(cfg.n, n_seed_groups * B, cfg.S, cfg.seed, dev,
                                   offsets=w.offsets)
    groups = [seeds_all[(g % n_seed_groups) * B:(g % n_seed_groups + 1) * B]
              for g in range(n_groups)]
    assert torch.equal(groups[0], w.seeds), "the first group must be the workload's group"

    # Buffers (outside the timed regions): sampling outputs at the per-batch
    # bounds dg_sample_bounds gives, packing outputs at the largest size any
    # group of the stream needs (a pre-pass samples and packs every group
    # without copying rows).
    node_cap, edge_cap = dg.sample_bounds(cfg.n, w.num_edges, cfg.S, fan)
    mem = torch.empty(cfg.n, dtype=torch.int64, device=dev)  # (node, batch) membership
    ws_s = torch.empty(dg._L.dg_sample_workspace_bytes(cfg.n, B, node_cap, edge_cap,
                                                       dg.sample_flags(direct=True)),
                       dtype=torch.uint8, device=dev)
    sr = dg.sample_group(w.offsets, w.indices, groups[0], fan, w.rng_seed, membership=mem,
                         workspace=ws_s, direct=True, node_cap=node_cap, edge_cap=edge_cap)
    pre = []
    ws_pre = None
    for g in range(n_groups):
        s_ = dg.sample_group(w.offsets, w.indices, groups[g], fan, w.rng_seed, batch_base=g * B,
                             out=sr, workspace=ws_s, membership=mem, direct=True)
        cnt_ = s_.node_count.copy()
        need_ws = dg._L.dg_pack_workspace_bytes(cfg.n, B, int(cnt_.sum()))
        if ws_pre is None or ws_pre.numel() < need_ws:
            ws_pre = torch.empty(need_ws, dtype=torch.uint8, device=dev)
        p_ = dg.pack_group(w.feats, w.cache_slot, s_.nodes, cnt_, membership=mem,
                           tables_only=True, workspace=ws_pre)
        pre.append({**s_.sizes, **{k: p_.sizes[k] for k in
                                   ("packed_rows", "unique_nodes", "unique_packed")}})
        del p_
    del ws_pre
    torch.cuda.empty_cache()
    max_rows = max(p["packed_rows"] for p in pre)
    max_total = max(p["total_nodes"] for p in pre)
    nmax = max(p["max_batch_nodes"] for p in pre)

    def pack_out():
        return dg.PackResult(
            packed=torch.empty((max(max_rows, 1), R), dtype=torch.uint8, device=dev),
            packed_ids=torch.empty(max(max_rows, 1), dtype=torch.int32, device=dev),
            packed_ptr=torch.empty(B + 1, dtype=torch.int64, device=dev),
            packed_ptr_host=np.zeros(B + 1, dtype=np.int64),
            loc=torch.empty((B, node_cap), dtype=torch.int32, device=dev), unique=None,
            sizes={}, timing=None, row_bytes=R)

    # `sets` packing output sets used in turn, so that step k never overwrites
    # what the assembly of an earlier step is still reading, and as many packing
    # workspaces, since in the pipelined region a packing call's row copy may
    # still be queued on the assembly stream when the next call starts; step k
    # waits only for the assembly of step k - sets
    n_sets = args.sets
    fused = not args.two_calls
    pr2 = [pack_out() for _ in range(n_sets)]
    ws_p2 = [torch.empty(dg._L.dg_sample_pack_workspace_bytes(cfg.n, B, node_cap) if fused else
                         dg._L.dg_pack_workspace_bytes(cfg.n, B, max_total), dtype=torch.uint8,
                         device=dev) for _ in range(n_sets)]
    # assembly output buffers used in turn: the library assembles up to ASM_GROUP
    # consecutive mini-batches with buffers of their own in one launch
    ybuf = [torch.empty((nmax, R), dtype=torch.uint8, device=dev) for _ in range(ASM_GROUP)]
    log(f"{n_groups} groups: pairs {min(p['total_nodes'] for p in pre):,}.."
        f"{max_total:,} edges {min(p['total_edges'] for p in pre):,}.."
        f"{max(p['total_edges'] for p in pre):,} packed rows up to {max_rows:,}")

    # Sampling and packing run on `stream` and return when their work is done;
    # the fan-out gather is timed by HIP events inside dg_pack_group.  Assembly
    # runs on `s_asm`: serially (the host waits for it) or pipelined, where
    # assembly of step k overlaps sampling and packing of step k+1 (both
    # streams at default priority).  In the pipelined region packing also leaves
    # its row copy (the fan-out gather) queued on s_asm ahead of the assembly
    # (DG_PACK_ROWS_STREAM), so the bandwidth-bound copy runs beside the next
    # step's sampling instead of on the sampling stream.  Each step's B
    # assembly launches are issued by one dg_assemble_batches call with that
    # step's own sizes; its host time is reported.
    s_asm = torch.cuda.Stream(device=dev)
    asm_done = [torch.cuda.Event() for _ in range(n_sets)]
    pack_done = [torch.cuda.Event() for _ in range(n_sets)]
    # timing events, created (by a first record) before any timed region
    nev = max(args.steps, args.warmup)
    ev_pool = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(nev)]
    for a_, b_ in ev_pool:
        a_.record(s_asm)
        b_.record(s_asm)
    for e_ in asm_done + pack_done:
        e_.record(s_asm)
    torch.cuda.synchronize()

    class Assembler:
        """Issues each pipelined step's assembly from a host thread of its own,
        as the trainer stage of the paper's pipeline (§5.3) consumes assembled
        batches while the next group is sampled: the main thread goes on to
        the next sampling call while the assembly launches are enqueued.  Steps are
        handed over in order; a packing output set (slot) is packed again only
        after the assembly that reads it has been enqueued."""

        def __init__(self):
            self.q = queue.Queue()
            self.free = [threading.Event() for _ in range(n_sets)]
            for f in self.free:
                f.set()
            self.err = None
            self.enqueue_s = []
            self.t = threading.Thread(target=self._loop, daemon=True)
            self.t.start()

        def _loop(self):
            while True:
                item = self.q.get()
                if item is None:
                    self.q.task_done()
                    return
                slot, p_out, counts, e0, e1 = item
                try:
                    t0 = time.perf_counter()
                    s_asm.wait_event(pack_done[slot])
                    e0.record(s_asm)
                    dg.assemble_batches(w.cache, p_out, counts, ybuf, stream=s_asm)
                    e1.record(s_asm)
                    asm_done[slot].record(s_asm)
                    self.enqueue_s.append(time.perf_counter() - t0)
                except BaseException as e:  # reported by the main thread
                    self.err = e
                finally:
                    self.free[slot].set()
                    self.q.task_done()

        def drain(self):
            self.q.join()
            if self.err is not None:
                raise self.err

        def close(self):
            self.q.put(None)
            self.t.join()

    asm_thread = None if args.asm_inline else Assembler()

    # Mask state across steps: each sampling call leaves its workspace state
    # clear (DG_SAMPLE_EXIT_CLEAR) and each packing call clears the membership
    # mask as it reads it (DG_PACK_CLEAR_MEMBERSHIP), so from the second step on
    # sampling is told both are clear (DG_SAMPLE_ENTRY_CLEAR) and skips its two
    # full-mask fills.  The first call on ws_s starts from unknown contents.
    clearing = not args.fill_masks
    state = {"clear": False}
    # sampling's last count pass marks the 8-node lines that hold a member, and
    # packing's count pass reads only those lines
    lines = (None if args.no_member_lines else
             torch.empty(dg.member_lines_bytes(cfg.n), dtype=torch.uint8, device=dev))
    samp_phases = {False: [], True: []}  # per region, with --sample-timing
    call_phases = []  # the library's phase times of each timed serial call

    def run(gs, pipelined, record):
        """One step per group index in gs; returns per-step host marks, gather
        times, assembly times (events) and the step's sizes."""
        marks, gather_ms, evs, steps = [], [], [], []
        for k, g in enumerate(gs):
            slot = k % n_sets
            t0 = time.perf_counter()
            # Sampling writes the cached nodes' address-table entries into this
            # step's packing set (pr2[slot].loc), so the assembly that last read
            # that set must have been enqueued (by the assembly thread) and run.
            threaded = pipelined and asm_thread is not None
            if threaded:
                asm_thread.free[slot].wait()
                asm_thread.free[slot].clear()
            stream.wait_event(asm_done[slot])
            entry_clear = clearing and state["clear"]
            state["clear"] = False
            handoff = not args.no_loc_handoff
            rows_async = pipelined and not args.rows_inline and not args.timed_pack
            if fused:
                # one call; a timed call runs its row copy inside it
                timed_call = record or args.timed_pack or args.sample_timing
                s_out, p_out = dg.sample_pack_group(
                    w.offsets, w.indices, groups[g], fan, w.rng_seed, w.feats, w.cache_slot,
                    batch_base=g * B, out=sr, pack_out=pr2[slot], workspace=ws_s,
                    pack_workspace=ws_p2[slot], membership=mem, direct=True, stream=stream,
                    exit_clear=clearing, entry_clear=entry_clear, timing=timed_call,
                    rows_stream=s_asm if (rows_async and not timed_call) else None)
                counts = s_out.node_count.copy()
                if args.sample_timing:
                    samp_phases[pipelined].append(dict(s_out.timing))
                t1 = t2 = time.perf_counter()
            else:
                s_out = dg.sample_group(w.offsets, w.indices, groups[g], fan, w.rng_seed,
                                        batch_base=g * B, out=sr, workspace=ws_s,
                                        membership=mem, direct=True, stream=stream,
                                        exit_clear=clearing, entry_clear=entry_clear,
                                        member_lines=lines, timing=args.sample_timing,
                                        cache_slot=w.cache_slot if handoff else None,
                                        loc=pr2[slot].loc if handoff else None)
                counts = s_out.node_count.copy()
                if args.sample_timing:
                    samp_phases[pipelined].append(dict(s_out.timing))
                t1 = time.perf_counter()
                p_out = dg.pack_group(w.feats, w.cache_slot, s_out.nodes, counts,
                                      out=pr2[slot], workspace=ws_p2[slot],
                                      timing=record or args.timed_pack, membership=mem,
                                      clear_membership=clearing, stream=stream,
                                      rows_stream=s_asm if rows_async else None,
                                      member_lines=lines, loc_pending=handoff)
                t2 = time.perf_counter()
            state["clear"] = clearing
            e0, e1 = ev_pool[k % nev]
            pack_done[slot].record(stream)
            if threaded:
                asm_thread.q.put((slot, p_out, counts, e0, e1))
            else:
                s_asm.wait_event(pack_done[slot])
                e0.record(s_asm)
                dg.assemble_batches(w.cache, p_out, counts, ybuf, stream=s_asm)
                e1.record(s_asm)
                asm_done[slot].record(s_asm)
            t3 = time.perf_counter()
            if not pipelined:
                e1.synchronize()
                evs.append(e0.elapsed_time(e1))
            marks.append((t1 - t0, t2 - t1, t3 - t2))
            steps.append({**s_out.sizes, **{k_: p_out.sizes[k_] for k_ in
                                            ("packed_rows", "unique_nodes", "unique_packed")},
                          # frontier entries over all hops: the nodes listed before
                          # the last hop's segment
                          "frontier": int(s_out.hop_ptr[:, len(fan)].sum())})
            if record:
                gather_ms.append(p_out.timing["gather_ms"])
                call_phases.append(dict(p_out.timing))
        if asm_thread is not None:
            asm_thread.drain()
        torch.cuda.synchronize()
        return marks, gather_ms, evs, steps

    def timed(gs, pipelined):
        run(gs[:args.warmup], pipelined, False)
        torch.cuda.synchronize()
        if asm_thread is not None:
            asm_thread.enqueue_s.clear()
        t_start = time.perf_counter()
        # per-phase timing (which runs the packing call's phases one after the
        # other) only in the serial region
        res = run(gs[args.warmup:], pipelined, not pipelined)
        torch.cuda.synchronize()
        t_total = time.perf_counter() - t_start
        for g, st in zip(gs[args.warmup:], res[3]):  # the pre-pass saw the same sizes
            if any(st[k] != pre[g][k] for k in ("total_nodes", "total_edges", "packed_rows")):
                raise RuntimeError(f"group {g}: sizes differ from the pre-pass")
        enq = list(asm_thread.enqueue_s) if (asm_thread is not None and pipelined) else []
        return (t_total,) + res + (enq,)

    def feature_bytes(st):
        """Feature bytes the method must move for one group: packing reads each
        non-cached unique row once and writes one row per packed row; assembly
        reads and writes one row per (node, batch) pair."""
        return R * (st["unique_packed"] + st["packed_rows"]), 2 * R * st["total_nodes"]

    # timed regions: K whole steps serially, then K whole steps pipelined, each
    # over groups of its own
    serial_groups = list(range(n_region))
    pipe_groups = list(range(n_region, 2 * n_region))
    t_serial, marks, gather_ms, asm_ms, steps_s, _ = timed(serial_groups, False)
    if args.no_pipeline:
        t_total, marks_p, steps_p, enq_p = t_serial, marks, steps_s, []
    else:
        t_total, marks_p, _, _, steps_p, enq_p = timed(pipe_groups, True)
    # secondary figure: the workload's own group repeated in every step (the
    # same index working set and hot rows each time), pipelined
    t_rep, _, _, _, steps_r, _ = timed([0] * n_region, not args.no_pipeline)
    if asm_thread is not None:
        asm_thread.close()
    samp_ms = [1e3 * m[0] for m in marks]
    pack_ms = [1e3 * m[1] for m in marks]

    Fp_s = [feature_bytes(st) for st in steps_s]
    F_pack_s = sum(a for a, _ in Fp_s)
    F_asm_s = sum(b for _, b in Fp_s)
    F_main = sum(sum(feature_bytes(st)) for st in steps_p)
    ms_step = 1e3 * t_total / args.steps
    value = F_main / t_total / 1e9
    device = device_info(dev)
    ms_serial = 1e3 * t_serial / args.steps
    # fan-out gather: one k_fanout16 launch per step, timed by the library's
    # HIP events on the call's stream (serial region)
    g_ms = float(np.mean(gather_ms))
    achieved = F_pack_s / (sum(gather_ms) * 1e-3) / 1e9
    # assembly: dg_assemble_batches runs ASM_GROUP consecutive mini-batches (with
    # output buffers of their own, one per ybuf entry) per k_assemble16_group launch;
    # its average launch time is the steps' assembly time (HIP events on its
    # stream, serial region) over the launches, and its bytes the steps'
    # assembly bytes over them
    asm_launches = (B + ASM_GROUP - 1) // ASM_GROUP
    a_ms = float(np.sum(asm_ms)) / (args.steps * asm_launches)
    F_asm_launch = F_asm_s / (args.steps * asm_launches)
    achieved_asm = F_asm_launch / (a_ms * 1e-3) / 1e9
    edges = sum(st["total_edges"] for st in steps_s)
    sizes_rep = steps_r[0]

    def span(key, steps):
        v = [st[key] for st in steps]
        return [min(v), max(v)] if min(v) != max(v) else v[0]

    out = {
        "metric": "packed+assembled feature GB/s (and % HBM peak); sampled edges/s, 1 MI355X",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "device": device,
        "config": {"workload": cfg.name, "nodes": cfg.n, "edges": w.num_edges,
                   "rmat_draws": cfg.draws, "feature": f"{cfg.dim}x{str(cfg.dtype)[6:]}",
                   "row_bytes": R, "batches": B, "seeds_per_batch": cfg.S, "fanouts": fan,
                   "cache_rows": int(w.cache_nodes.numel()), "parallelism": "single-gpu"},
        "frac_hbm_peak": round(value / HBM_PEAK_GBPS, 4),
        "groups": (f"a stream of distinct groups: every step samples, packs and assembles a group "
                   f"of its own ({B} mini-batches x {cfg.S} seeds, consecutive groups of one "
                   f"seed stream drawn without replacement, global batch numbers g*{B}..); "
                   f"value = the timed steps' own feature bytes over their wall time"
                   + ("" if n_seed_groups == n_groups else
                      f"; the graph has seed candidates for {n_seed_groups} disjoint groups, "
                      f"so the {n_groups} groups reuse those seed sets in turn")),
        "seed_groups": n_seed_groups,
        "pipelined": ("no: --no-pipeline, value is the serial rate" if args.no_pipeline else
                      "assembly of step k (second stream) overlaps sampling and packing of "
                      "step k+1; the serial figures below wait for each step's assembly"),
        "packing_sets": n_sets,
        "assembly_issue": (f"direct calls: one dg_assemble_batches call (B/{ASM_GROUP} launches "
                           f"of {ASM_GROUP} mini-batches) per step, "
                           + ("issued by the main thread" if asm_thread is None else
                              "issued by a host thread of its own in the pipelined region "
                              "(the trainer side), by the main thread in the serial region")),
        "sample_pack": ("one dg_sample_pack_group call per step: the last hop's compaction "
                        "pass also does packing's pass over the membership words, and the "
                        "address tables of non-cached entries follow from one kernel"
                        if fused else "dg_sample_group, then dg_pack_group"),
        "pack_rows": ("pipelined region: packing's row copy queued on the assembly stream "
                      "(DG_PACK_ROWS_STREAM)" if not (args.rows_inline or args.timed_pack
                                                      or args.no_pipeline)
                      else "inside the packing call"),
        "address_tables": ("sampling writes the cached nodes' entries as it lists them, the "
                           "others come from the fused pass's packed rows" if fused else
                           "sampling writes the cached nodes' entries as it lists them; "
                           "packing completes the others (DG_PACK_LOC_PENDING)"
                           if not args.no_loc_handoff else "built by packing alone"),
        "member_lines": ("not needed: packing's pass is the last hop's sweep of every word"
                         if fused else
                         "packing reads only the membership lines sampling marked"
                         if lines is not None else "packing reads every membership word"),
        "mask_clearing": ("clearing flags: packing clears the membership words it reads and "
                          "sampling leaves its state clear, so no full-mask fill runs per step"
                          if clearing else "two full-mask fills in every sampling call"),
        "serial": {"ms_per_step": round(ms_serial, 3),
                   "value": round((F_pack_s + F_asm_s) / t_serial / 1e9, 2)},
        "repeated_group": {"what": "the workload's group sampled, packed and assembled in every "
                                   "step (same seeds each time)",
                           "ms_per_step": round(1e3 * t_rep / args.steps, 3),
                           "value": round(args.steps * sum(feature_bytes(sizes_rep)) / t_rep
                                          / 1e9, 2)},
        "pipelined_phases_ms": {**({"sample_and_pack_call": round(1e3 * float(np.mean(
                                        [m[0] for m in marks_p])), 3)} if fused else
                                     {"sample": round(1e3 * float(np.mean(
                                         [m[0] for m in marks_p])), 3),
                                      "pack": round(1e3 * float(np.mean(
                                          [m[1] for m in marks_p])), 3)}),
                                "host_enqueue_assembly": round(1e3 * float(np.mean(
                                    enq_p or [m[2] for m in marks_p])), 3),
                                "host_enqueue_assembly_on": ("the assembly thread"
                                                             if asm_thread is not None
                                                             else "the main thread")},
        "sampled_edges_per_s": round(edges / ((np.sum(samp_ms) - (np.sum(gather_ms) if fused
                                                                  else 0.0)) * 1e-3), 1),
        "sampled_edges_per_s_over": ("the sample-and-pack call less its row copy (sampling "
                                     "with packing's tables folded into its last pass; serial "
                                     "region)" if fused else "the sampling call (serial region)"),
        "phases_ms": {**({"sample_and_pack_call": round(float(np.mean(samp_ms)), 3)} if fused
                         else {"sample": round(float(np.mean(samp_ms)), 3),
                               "pack": round(float(np.mean(pack_ms)), 3)}),
                      "fanout_gather": round(g_ms, 3),
                      "assemble_all_batches": round(float(np.mean(asm_ms)), 3),
                      "host_enqueue_assembly": round(
                          1e3 * float(np.mean([m[2] for m in marks])), 3)},
        "paper_context": {
            "what": ("the paper gives no kernel-level figure for this path (so vs_baseline is "
                     "null); its whole pre-processing of ogbn-papers100M (cache configuration "
                     "and batched packing, 52.9 GB of fp32 features) took about 0.03 h (Tables "
                     "1 and 2), which puts it near 0.5 GB/s (derived), bound by an NVMe SSD of "
                     "3 GB/s on an AMD EPYC 7R32 host with one NVIDIA A10G (the platform of "
                     "§7, Table 4)"),
            "preprocessing_GBps": 0.5},
        "call_phases_ms": {
            "what": ("the library's HIP-event phases of each timed serial call, median: draws "
                     "(all hops), compaction (with one call, the last hop's pass also does "
                     "packing's), relabelling, packing's own passes (two calls, or where they "
                     "are not fused), address tables, row copy"),
            **{k.replace("_ms", ""): round(_median([t[k] for t in call_phases]), 3)
               for k in ("sample_ms", "dedup_ms", "relabel_ms", "mark_ms", "order_ms",
                         "loc_ms", "gather_ms", "total_ms")}} if call_phases else None,
        "implied_line_rate": ({
            "what": ("64-byte lines the draw phase touches at random: one CSR index line and "
                     "one membership-word line per sampled edge, one offsets line per frontier "
                     "entry; over the draw phase's own time (the library's HIP events, median "
                     "of the timed serial calls)"),
            "lines_per_step": int(np.median([2 * st["total_edges"] + st["frontier"]
                                             for st in steps_s])),
            "lines_per_s": round(np.median([2 * st["total_edges"] + st["frontier"]
                                            for st in steps_s])
                                 / (_median([t["sample_ms"] for t in call_phases]) * 1e-3),
                                 1)} if call_phases and fused else None),
        "phase_gbps": {**({} if fused else
                          {"pack_call": round(F_pack_s / (np.sum(pack_ms) * 1e-3) / 1e9, 1)}),
                       "assemble_calls": round(F_asm_s / (np.sum(asm_ms) * 1e-3) / 1e9, 1)},
        "sizes": {k: span(k, steps_p) for k in
                  ("total_nodes", "total_edges", "packed_rows", "unique_nodes",
                   "unique_packed")},
        # the dominant kernel by time: batch assembly (B/4 launches per step)
        "roofline": {"kernel": f"k_assemble16_group (batch assembly, {ASM_GROUP} mini-batches "
                               "per launch)",
                     "bound": "hbm", "achieved": round(achieved_asm, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved_asm / HBM_PEAK_GBPS, 4),
                     "traffic": load_traffic(cfg.name, "assemble"),
                     "algorithmic_bytes": int(round(F_asm_launch)),
                     "launch_ms": round(a_ms, 4), "launches_per_step": asm_launches},
        # the other row kernel: packing's fan-out gather (one launch per step)
        "roofline_fanout": {"kernel": "k_fanout16 (fan-out gather)", "bound": "hbm",
                            "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                            "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                            "traffic": load_traffic(cfg.name, "fanout_gather"),
                            "algorithmic_bytes": int(round(F_pack_s / args.steps)),
                            "launch_ms": round(g_ms, 4), "launches_per_step": 1},
    }

    if args.copy_calib:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    if args.sample_timing:
        keys = ("sample_ms", "dedup_ms", "relabel_ms", "total_ms")
        out["sampling_phases_ms"] = {
            name: {k.replace("_ms", ""): round(_median([t[k] for t in v[-args.steps:]]), 3)
                   for k in keys}
            for name, v in (("serial", samp_phases[False]), ("pipelined", samp_phases[True]))
            if v}
    if not args.no_ceiling:
        # what a plain copy of rows reaches on this machine, outside the timed
        # regions: the row kernels' fraction of 8 TB/s is read against it
        c = experiment_ceiling(dg, w, cfg, 3)
        out["row_copy_ceiling"] = {
            "kind": "dg_gather_rows of 2 GiB of this workload's rows, same process",
            "unit": "GB/s",
            "random_rows": c["cases"]["random_over_table"]["GBps"],
            "in_order": c["cases"]["in_order"]["GBps"],
            "assembly_achieved_over_in_order": round(
                out["roofline"]["achieved"] / c["cases"]["in_order"]["GBps"], 3)}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, cfg, args.cpu_batches or cfg.B)
    print(json.dumps(out), flush=True)


def _median(v):
    v = sorted(v)
    return v[len(v) // 2]


def experiment_pack_ab(dg, w, cfg, reps):
    """Batched packing (one fan-out gather that reads each non-cached row once)
    against individual packing (one gather per mini-batch, a row read per
    mini-batch that needs it), on the same packing tables; paper §5.2, Fig. 6,
    Fig. 17."""
    import torch
    R, B = cfg.row_bytes, cfg.B
    mem = torch.empty(cfg.n, dtype=torch.int64, device="cuda")
    sr = dg.sample_group(w.offsets, w.indices, w.seeds, list(cfg.fanouts), w.rng_seed,
                         membership=mem)
    pr = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count, membership=mem)
    buf = torch.empty_like(pr.packed)
    # Individual packing is B launches.  Issued call by call from Python, the
    # GPU can wait on the host between them, so its time is taken from a
    # captured HIP graph of the B launches (the eager time is reported too).
    s_cap = torch.cuda.Stream()
    s_cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s_cap):
        dg.pack_individual(w.feats, pr.packed_ids, pr.packed_ptr_host, buf)
    torch.cuda.current_stream().wait_stream(s_cap)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        dg.pack_individual(w.feats, pr.packed_ids, pr.packed_ptr_host, buf)
    torch.cuda.synchronize()
    t_b, t_i, t_e = [], [], []
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for _ in range(reps + 1):
        p = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count, out=pr,
                          membership=mem, timing=True)
        t_b.append(p.timing["gather_ms"])
        buf.zero_()
        ev[0].record()
        graph.replay()
        ev[1].record()
        ev[1].synchronize()
        t_i.append(ev[0].elapsed_time(ev[1]))
        ev[0].record()
        dg.pack_individual(w.feats, pr.packed_ids, pr.packed_ptr_host, buf)
        ev[1].record()
        ev[1].synchronize()
        t_e.append(ev[0].elapsed_time(ev[1]))
    rows = pr.sizes["packed_rows"]
    same = bool(torch.equal(buf[:rows], pr.packed[:rows]))  # call by call
    buf.zero_()
    graph.replay()
    torch.cuda.synchronize()
    same = same and bool(torch.equal(buf[:rows], pr.packed[:rows]))  # graph replay
    Uc = pr.sizes["unique_packed"]
    tb, ti, te = _median(t_b[1:]), _median(t_i[1:]), _median(t_e[1:])
    return {"experiment": "batched vs individual packing (row copy only)", "workload": cfg.name,
            "cache_rows": int(w.cache_nodes.numel()), "row_bytes": R, "batches": B,
            "packed_rows": rows, "unique_packed": Uc,
            "batched": {"ms": round(tb, 3), "row_reads": Uc,
                        "bytes": R * (Uc + rows), "GBps": round(R * (Uc + rows) / tb / 1e6, 1)},
            "individual": {"ms": round(ti, 3), "row_reads": rows, "launches": B,
                           "issue": "replay of a captured HIP graph of the launches",
                           "bytes": 2 * R * rows, "GBps": round(2 * R * rows / ti / 1e6, 1),
                           "ms_issued_call_by_call": round(te, 3)},
            "speedup": round(ti / tb, 3), "read_ratio": round(rows / max(Uc, 1), 3),
            "identical_output": same}


def experiment_cache_fill(dg, w, cfg, reps):
    """The cache filled by batched packing as one more mini-batch (§5.2): one
    packing call whose fan-out gather also writes the cache table, against the
    same packing call followed by a separate row gather of the cache
    (dg_gather_rows over cache_nodes).  Times are the gather launches' own
    (the library's HIP events for the packing gather, events around
    dg_gather_rows), median over reps."""
    import torch
    R, B = cfg.row_bytes, cfg.B
    C = int(w.cache_nodes.numel())
    nodes = w.cache_nodes.to(torch.int32)
    mem = torch.empty(cfg.n, dtype=torch.int64, device="cuda")
    sr = dg.sample_group(w.offsets, w.indices, w.seeds, list(cfg.fanouts), w.rng_seed,
                         membership=mem, direct=True)
    table = torch.empty((C, R), dtype=torch.uint8, device="cuda")
    pr = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count, membership=mem)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    one, two_pack, two_cache = [], [], []
    for _ in range(reps + 1):
        p = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count, out=pr,
                          membership=mem, timing=True, cache_nodes=nodes, cache_table=table)
        one.append(p.timing["gather_ms"])
        p = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count, out=pr,
                          membership=mem, timing=True)
        two_pack.append(p.timing["gather_ms"])
        ev[0].record()
        dg.gather_rows(w.feats, nodes, out=table)
        ev[1].record()
        ev[1].synchronize()
        two_cache.append(ev[0].elapsed_time(ev[1]))
    ok = bool(torch.equal(table[:1024], w.feats.index_select(0, w.cache_nodes[:1024])
                          .view(torch.uint8).reshape(-1, R)))
    Uc, rows = pr.sizes["unique_packed"], pr.sizes["packed_rows"]
    t1 = _median(one[1:])
    t2 = _median(two_pack[1:]) + _median(two_cache[1:])
    bytes_ = R * (Uc + rows) + 2 * R * C
    return {"experiment": "cache filled by the packing gather vs a separate gather",
            "workload": cfg.name, "cache_rows": C, "row_bytes": R, "batches": B,
            "packed_rows": rows, "unique_packed": Uc, "bytes": bytes_,
            "one_launch": {"ms": round(t1, 3), "GBps": round(bytes_ / t1 / 1e6, 1)},
            "two_launches": {"ms": round(t2, 3), "GBps": round(bytes_ / t2 / 1e6, 1),
                             "pack_gather_ms": round(_median(two_pack[1:]), 3),
                             "cache_gather_ms": round(_median(two_cache[1:]), 3)},
            "speedup": round(t2 / t1, 3), "cache_table_checked": ok}


def experiment_cache(dg, w, cfg, reps):
    """Cache by access frequency (popcount of the group's membership words;
    §3, §4) against cache by in-degree, same size: packed rows and pack time."""
    import torch
    B = cfg.B
    C = int(w.cache_nodes.numel())
    mem = torch.empty(cfg.n, dtype=torch.int64, device="cuda")
    sr = dg.sample_group(w.offsets, w.indices, w.seeds, list(cfg.fanouts), w.rng_seed,
                         membership=mem)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    t_sel = []
    for _ in range(reps + 1):
        ev[0].record()
        slot_f, nodes_f, cached = dg.cache_by_frequency(mem, B, C)
        ev[1].record()
        ev[1].synchronize()
        t_sel.append(ev[0].elapsed_time(ev[1]))
    cache_f = dg.gather_rows(w.feats, nodes_f[:cached])
    res = {}
    for name, slot in (("in_degree", w.cache_slot), ("frequency", slot_f)):
        ts = []
        for _ in range(reps + 1):
            p = dg.pack_group(w.feats, slot, sr.nodes, sr.node_count, membership=mem, timing=True)
            ts.append(p.timing["total_ms"])
        res[name] = {"packed_rows": p.sizes["packed_rows"], "unique_packed": p.sizes["unique_packed"],
                     "pack_ms": round(_median(ts[1:]), 3)}
    accesses = sr.sizes["total_nodes"]
    return {"experiment": "cache by access frequency vs by in-degree", "workload": cfg.name,
            "cache_rows": C, "cached": cached, "accesses": accesses,
            "select_ms": round(_median(t_sel[1:]), 3), "cache_table_bytes": int(cache_f.numel()),
            "in_degree": res["in_degree"], "frequency": res["frequency"],
            "hit_share": {k: round(1 - v["packed_rows"] / accesses, 4) for k, v in res.items()}}


def experiment_layered(dg, w, cfg, reps):
    """Sampling with the paper's frontier rule (only newly reached nodes sample
    next, Fig. 1) against the layer-wise rule (every node so far samples)."""
    res = {}
    for name, layered in (("new_nodes", False), ("layered", True)):
        sr = dg.sample_group(w.offsets, w.indices, w.seeds, list(cfg.fanouts), w.rng_seed,
                             layered=layered, direct=True)
        ts = []
        for _ in range(reps + 1):
            t0 = time.perf_counter()
            dg.sample_group(w.offsets, w.indices, w.seeds, list(cfg.fanouts), w.rng_seed,
                            out=sr, layered=layered, direct=True)
            ts.append(time.perf_counter() - t0)
        t = _median(ts[1:])
        res[name] = {"ms": round(1e3 * t, 3), "edges": sr.sizes["total_edges"],
                     "nodes": sr.sizes["total_nodes"],
                     "edges_per_s": round(sr.sizes["total_edges"] / t, 1)}
    return {"experiment": "sampling frontier rule", "workload": cfg.name, "fanouts":
            list(cfg.fanouts), "batches": cfg.B, **res}


def experiment_minhash(dg, w, cfg, reps, k=4, page_bytes=4096):
    """Disk-cache reordering by MinHash (§5.1, Alg. 1): the non-cached nodes the
    group requires form the disk cache V_d; count the 4 KiB pages each
    mini-batch touches when V_d is laid out in ID order and in MinHash order."""
    import torch
    B, R = cfg.B, cfg.row_bytes
    rpp = max(1, page_bytes // R)  # rows per page
    mem = torch.empty(cfg.n, dtype=torch.int64, device="cuda")
    sr = dg.sample_group(w.offsets, w.indices, w.seeds, list(cfg.fanouts), w.rng_seed,
                         membership=mem)
    accessed = (mem != 0).nonzero().squeeze(1)
    vd = accessed[w.cache_slot[accessed] < 0].to(torch.int32).contiguous()  # ascending IDs
    g = torch.Generator().manual_seed(cfg.seed + 1)
    perms = torch.stack([torch.randperm(B, generator=g) for _ in range(k)]).to(torch.int32).cuda()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ts = []
    for _ in range(reps + 1):
        ev[0].record()
        order, sig = dg.minhash_order(mem, B, vd, perms)
        ev[1].record()
        ev[1].synchronize()
        ts.append(ev[0].elapsed_time(ev[1]))

    def pages(layout):
        pos = torch.full((cfg.n,), -1, dtype=torch.int64, device="cuda")
        pos[layout.long()] = torch.arange(layout.numel(), device="cuda")
        total = 0
        for b in range(B):
            p = pos[sr.batch_nodes(b).long()]
            p = p[p >= 0] // rpp
            total += int(torch.unique(p).numel())
        return total

    lower = sum(-(-int((pos_b := w.cache_slot[sr.batch_nodes(b).long()] < 0).sum()) // rpp)
                for b in range(B))
    id_pages, mh_pages = pages(vd), pages(order)
    return {"experiment": "disk-cache pages touched, ID order vs MinHash order",
            "workload": cfg.name, "disk_cache_entries": int(vd.numel()), "hash_functions": k,
            "rows_per_page": rpp, "order_ms": round(_median(ts[1:]), 3),
            "pages_id_order": id_pages, "pages_minhash_order": mh_pages,
            "pages_lower_bound": lower, "reduction": round(id_pages / max(mh_pages, 1), 3)}


def _popcount64(x):
    """Set bits of each int64 word (SWAR; masks keep arithmetic shifts exact)."""
    x = x - ((x >> 1) & 0x5555555555555555)
    x = (x & 0x3333333333333333) + ((x >> 2) & 0x3333333333333333)
    x = (x + (x >> 4)) & 0x0F0F0F0F0F0F0F0F
    return ((x * 0x0101010101010101) >> 56) & 0xFF


# Node access distribution reported by the paper (Table 3), per dataset:
# access share of the nodes ranked <1%, 1-5%, 5-10%, >10% by access frequency.
PAPER_TABLE3 = {"FS": [14.1, 25.5, 18.2, 42.1], "PS": [43.2, 36.5, 11.2, 9.1],
                "MG": [56.4, 32.3, 7.3, 4.0], "IG": [22.5, 30.0, 20.8, 26.7]}


def experiment_ceiling(dg, w, cfg, reps, out_bytes=2 << 30):
    """What a row copy can reach on this memory system, to read the row
    kernels' fraction of the 8 TB/s peak against: the library's plain row
    gather (dg_gather_rows, the same 16-byte row machinery as the fan-out
    gather and the assembly) of about out_bytes (at least 2M rows) from the
    workload's feature table,
    with ids drawn uniformly over the whole table, over the first C rows (the
    size of the cache table the assembly reads; only with a cache) and in order
    (a streaming copy); and, for comparison, the runtime's own device-to-device
    copy (2 * row_bytes * n_rows bytes, like the gathers: each row read once and
    written once), fill (writes only) and fp32 sum (reads only) of the in-order
    rows (row_bytes * n_rows bytes each)."""
    import torch
    R = cfg.row_bytes
    N = w.feats.shape[0]
    C = int(w.cache_nodes.numel())
    n = min(max(1 << 21, out_bytes // R), N)
    dev = w.feats.device
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg.seed + 7)
    cases = {"random_over_table": torch.randint(0, N, (n,), generator=gen, device=dev,
                                                dtype=torch.int32)}
    if C > 0:
        cases["random_over_cache_rows"] = torch.randint(0, min(C, N), (n,), generator=gen,
                                                        device=dev, dtype=torch.int32)
    cases["in_order"] = torch.arange(n, dtype=torch.int32, device=dev)
    out = torch.empty((n, R), dtype=torch.uint8, device=dev)
    table = w.feats.view(torch.uint8).view(N, R)
    src = table[:n]  # the in-order rows, for the runtime's copy
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    nbytes = 2 * R * n

    def timed(fn, batch=10):
        # back-to-back launches between one pair of events, so that the host's
        # time to issue a call is hidden behind the previous one
        t = []
        fn()
        torch.cuda.synchronize()
        for _ in range(reps):
            ev[0].record()
            for _ in range(batch):
                fn()
            ev[1].record()
            ev[1].synchronize()
            t.append(ev[0].elapsed_time(ev[1]) / batch)
        return _median(t)

    res = {}
    for name, ids in cases.items():
        ms = timed(lambda: dg.gather_rows(w.feats, ids, out=out))
        ok = bool(torch.equal(out[:1024], table.index_select(0, ids[:1024].long())))
        res[name] = {"ms": round(ms, 4), "bytes": nbytes, "GBps": round(nbytes / ms / 1e6, 1),
                     "checked": ok}
    ms = timed(lambda: out.copy_(src))
    res["runtime_device_copy"] = {"ms": round(ms, 4), "bytes": nbytes,
                                  "GBps": round(nbytes / ms / 1e6, 1)}
    # the runtime's write-only fill and read-only reduction of the same rows
    ms = timed(lambda: out.fill_(1))
    res["runtime_fill"] = {"ms": round(ms, 4), "bytes": R * n, "GBps": round(R * n / ms / 1e6, 1)}
    words = src.view(torch.float32)  # the rows' bytes as fp32 words: only the read is timed
    ms = timed(lambda: words.sum())
    res["runtime_sum"] = {"ms": round(ms, 4), "bytes": R * n, "GBps": round(R * n / ms / 1e6, 1)}
    return {"experiment": "row copy ceilings (dg_gather_rows and the runtime's copy)",
            "workload": cfg.name, "row_bytes": R, "rows": n, "table_rows": N, "cache_rows": C,
            "reps": reps, "peak_GBps": HBM_PEAK_GBPS, "cases": res}


def experiment_regime(dg, w, cfg, reps, groups=16):
    """Regime check of the synthetic workload: sample `groups` consecutive
    groups of B mini-batches (about an epoch's seeds for L100), count each
    node's accesses (the mini-batches that require it), rank nodes by count and
    report the access share of the top <1%, 1-5%, 5-10% and >10% of nodes, next
    to the paper's Table 3; also sum|P_b| / N per group and over all groups
    (packed rows relative to the feature table, at the workload's cache)."""
    import torch

    import synth
    B, N = cfg.B, cfg.n
    dev = w.offsets.device
    seeds = synth.seed_batches(N, groups * B, cfg.S, cfg.seed, dev, offsets=w.offsets)
    assert torch.equal(seeds[:B], w.seeds), "the first group must be the benchmark group"
    cnt = torch.zeros(N, dtype=torch.int32, device=dev)
    mem = torch.empty(N, dtype=torch.int64, device=dev)
    packed_rows = []
    for g in range(groups):
        sr = dg.sample_group(w.offsets, w.indices, seeds[g * B:(g + 1) * B].contiguous(),
                             list(cfg.fanouts), w.rng_seed, batch_base=g * B, membership=mem,
                             direct=True)
        cnt += _popcount64(mem).to(torch.int32)
        pr = dg.pack_group(w.feats, w.cache_slot, sr.nodes, sr.node_count, membership=mem,
                           tables_only=True)
        packed_rows.append(pr.sizes["packed_rows"])
        del sr, pr
    total = int(cnt.sum(dtype=torch.int64))
    ranked = torch.sort(cnt, descending=True).values.to(torch.int64)
    cuts = [0, N // 100, N // 20, N // 10, N]
    shares = [round(100.0 * int(ranked[a:b].sum()) / total, 1) for a, b in zip(cuts, cuts[1:])]
    return {"experiment": "node access distribution (regime check)", "workload": cfg.name,
            "groups": groups, "mini_batches": groups * B, "seeds": groups * B * cfg.S,
            "accesses": total, "accessed_nodes": int((cnt > 0).sum()),
            "share_pct_by_rank": {"<1%": shares[0], "1-5%": shares[1], "5-10%": shares[2],
                                  ">10%": shares[3]},
            "paper_table3_pct": PAPER_TABLE3,
            "packed_rows_over_N": {"first_group": round(packed_rows[0] / N, 4),
                                   "all_groups": round(sum(packed_rows) / N, 4)},
            "cache_rows": int(w.cache_nodes.numel())}


def device_info(dev) -> dict:
    """The GPU, the ROCm and HIP versions, and its peak engine and memory clocks
    (the HIP runtime's device attributes; None where unavailable)."""
    import ctypes

    import torch
    props = torch.cuda.get_device_properties(dev)
    info = {"name": torch.cuda.get_device_name(dev), "arch": props.gcnArchName,
            "compute_units": props.multi_processor_count, "hip": torch.version.hip,
            "rocm": None, "peak_sclk_mhz": None, "peak_mclk_mhz": None}
    try:
        with open("/opt/rocm/.info/version") as f:
            info["rocm"] = f.read().strip()
    except OSError:
        pass
    try:
        hip = ctypes.CDLL("libamdhip64.so")
        idx = torch.device(dev).index or 0
        # hipDeviceAttributeClockRate = 5, hipDeviceAttributeMemoryClockRate = 60 (kHz)
        for key, attr in (("peak_sclk_mhz", 5), ("peak_mclk_mhz", 60)):
            v = ctypes.c_int(0)
            if hip.hipDeviceGetAttribute(ctypes.byref(v), attr, idx) == 0:
                info[key] = v.value // 1000
    except OSError:
        pass
    return info


def cpu_model() -> str:
    """The host CPU's model name, as lscpu reports it."""
    import subprocess
    try:
        txt = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for ln in txt.splitlines():
            if ln.startswith("Model name:"):
                return ln.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            return next((ln.split(":", 1)[1].strip() for ln in f
                         if ln.startswith("model name")), "unknown")
    except OSError:
        return "unknown"


def _oracle_pass(oracle, off, idx, X, slot, cache, seeds, fan, rng, batch_base, R, threads):
    """One group through the oracle: sampling, packing and assembly, timed per
    phase.  With threads > 1 each phase runs on runs of consecutive mini-batches
    in that many host threads: sampling is independent per mini-batch (draws are
    keyed by the global batch number), and a mini-batch's packed chunk, packed
    order and address table depend on its own node list only, so packing a run
    of batches gives the same per-batch outputs as packing the whole group.
    Returns (seconds per phase, sampled lists, packing results, their batch
    runs)."""
    from concurrent.futures import ThreadPoolExecutor
    nb = seeds.shape[0]
    cuts = [nb * t // threads for t in range(threads + 1)]
    t1 = time.perf_counter()
    rs = oracle.sample_group(off, idx, seeds, fan, rng, batch_base=batch_base, threads=threads)
    t2 = time.perf_counter()
    if threads == 1:
        parts = [oracle.pack_group(X, slot, rs["nodes"], with_unique=False)]
        runs = [(0, nb)]
    else:
        runs = [(cuts[t], cuts[t + 1]) for t in range(threads) if cuts[t + 1] > cuts[t]]
        with ThreadPoolExecutor(len(runs)) as ex:
            parts = list(ex.map(lambda r: oracle.pack_group(X, slot, rs["nodes"][r[0]:r[1]],
                                                            with_unique=False), runs))
    t3 = time.perf_counter()

    def assemble(i):
        rp, (lo_b, hi_b) = parts[i], runs[i]
        for b in range(hi_b - lo_b):
            lo, hi = rp["packed_ptr"][b], rp["packed_ptr"][b + 1]
            oracle.assemble_batch(cache, rp["packed"][lo:hi], rp["loc"][b], R)

    if threads == 1:
        assemble(0)
    else:
        with ThreadPoolExecutor(len(runs)) as ex:
            list(ex.map(assemble, range(len(runs))))
    t4 = time.perf_counter()
    return {"sample": t2 - t1, "pack": t3 - t2, "assemble": t4 - t3}, rs, parts, runs


def _group_bytes(rs, slot, R):
    """Algorithmic feature bytes of one group (the GPU's definition)."""
    import numpy as np
    allnodes = np.concatenate(rs["nodes"])
    u = np.unique(allnodes)
    unc = int((slot[u] < 0).sum())
    packed = int((slot[allnodes] < 0).sum())
    return R * (unc + packed) + 2 * R * allnodes.size, sum(len(x) for x in rs["edge_src"])


def cpu_baseline(w, cfg, nb, groups=2, small=True):
    """The oracle (single-threaded C, as it stands) timed on the host on a
    bounded sample of the same workload: the first `nb` mini-batches of
    `groups` consecutive groups of the seed stream (the benchmark's first groups),
    on the full graph and feature table, run on the host's cores (runs of
    mini-batches in parallel threads, at most 16: the host share of one GPU);
    beside it the same oracle on one core over the first group, and on one core
    over the small workloads T and M1."""
    import numpy as np
    import torch

    import oracle
    import synth

    threads = oracle.host_threads()
    if w.feats.numel() * w.feats.element_size() > (96 << 30):
        return {"skipped": "feature table above 96 GB: not copied to host memory"}
    t0 = time.perf_counter()
    log("cpu baseline: copying graph and features to host")
    off = w.offsets.cpu().numpy()
    idx = w.indices.cpu().numpy()
    B = cfg.B
    all_seeds = synth.seed_batches(cfg.n, groups * B, cfg.S, cfg.seed, w.offsets.device,
                                   offsets=w.offsets)
    assert torch.equal(all_seeds[:B], w.seeds), "the first group must be the benchmark group"
    all_seeds = all_seeds.cpu().numpy()
    X = w.feats.cpu().numpy()
    slot = w.cache_slot.cpu().numpy()
    cache = w.cache.cpu().numpy()
    R = cfg.row_bytes
    fan = list(cfg.fanouts)
    log(f"host copies in {time.perf_counter() - t0:.1f}s; oracle on {groups} x {nb} batches in "
        f"{threads} threads, then 1 x {nb} batches on one core")

    def measure(ngroups, nthreads):
        secs = {"sample": 0.0, "pack": 0.0, "assemble": 0.0}
        F = edges = 0
        for g in range(ngroups):
            s, rs, _, _ = _oracle_pass(oracle, off, idx, X, slot, cache,
                                       all_seeds[g * B:g * B + nb], fan, w.rng_seed, g * B, R,
                                       nthreads)
            for k in secs:
                secs[k] += s[k]
            f, e = _group_bytes(rs, slot, R)
            F += f
            edges += e
            del rs
        total = sum(secs.values())
        return {"value": round(F / total / 1e9, 4), "seconds": {k: round(v, 3)
                                                                for k, v in secs.items()},
                "sampled_edges_per_s": round(edges / secs["sample"], 1)}

    multi = measure(groups, threads)
    one = measure(1, 1)
    what = "the whole group" if nb == cfg.B else f"the first {nb} of {cfg.B} mini-batches"
    out = {"value": multi["value"], "unit": "GB/s", "cores": threads, "kind": "oracle",
           "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
           "sample": f"{what}, for {groups} consecutive groups of {cfg.name} (the benchmark's "
                     f"first groups of the seed stream; full graph and feature table on the "
                     f"host): sample + pack + assemble, one pass each, runs of mini-batches in "
                     f"{threads} host threads (the oracle itself is single-threaded C)",
           "seconds": multi["seconds"], "sampled_edges_per_s": multi["sampled_edges_per_s"],
           "one_core": {"value": one["value"], "unit": "GB/s", "cores": 1,
                        "sample": f"{what}, first group only",
                        "seconds": one["seconds"],
                        "sampled_edges_per_s": one["sampled_edges_per_s"]}}
    del X, off, idx
    if small:
        out["one_core_small"] = {}
        for name in ("T", "M1"):
            ws_ = synth.make_workload(name, device=w.offsets.device)
            c_ = ws_.cfg
            o_, i_ = ws_.offsets.cpu().numpy(), ws_.indices.cpu().numpy()
            X_, sl_, ca_ = ws_.feats.cpu().numpy(), ws_.cache_slot.cpu().numpy(), \
                ws_.cache.cpu().numpy()
            times = []
            for _ in range(3):  # the median of 3 runs
                s, rs, _, _ = _oracle_pass(oracle, o_, i_, X_, sl_, ca_,
                                           ws_.seeds.cpu().numpy(), list(c_.fanouts),
                                           ws_.rng_seed, 0, c_.row_bytes, 1)
                times.append(s)
            s = sorted(times, key=lambda x: sum(x.values()))[1]
            tot = sum(s.values())
            f, e = _group_bytes(rs, sl_, c_.row_bytes)
            out["one_core_small"][name] = {"value": round(f / tot / 1e9, 4), "unit": "GB/s",
                                           "seconds": {k: round(v, 4) for k, v in s.items()},
                                           "sampled_edges_per_s": round(e / s["sample"], 1)}
            del ws_, X_
    return out


if __name__ == "__main__":
    main()
