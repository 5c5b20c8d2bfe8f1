"""CPU oracle for the offline-sampling path — TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library
(``paper_2405_05231_amd``) never imports it and shares no code with it.

The arithmetic lives in ``oracle.c`` (plain C, single thread, qsort/bsearch,
written from the paper: node-wise sampling §2 Fig. 1, batched packing §5.2
Fig. 6b, address tables §6, feature assembling §4 Fig. 3).  This module only
compiles it with gcc and marshals numpy arrays in and out.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

I64P = ctypes.POINTER(ctypes.c_int64)
I32P = ctypes.POINTER(ctypes.c_int32)
VP = ctypes.c_void_p


# A test may load another build of the oracle (a sanitizer build, or a copy with
# a planted mistake) by naming its shared library here.
LIB_ENV = "DG_ORACLE_LIB"


def compile_oracle(out: str, src: str = _SRC, extra=()) -> str:
    """gcc build of an oracle source into the shared library `out`."""
    tmp = out + ".tmp"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Werror", *extra,
                    src, "-o", tmp], check=True)
    os.replace(tmp, out)
    return out


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so with gcc (no GPU code involved)."""
    if force or not os.path.exists(_LIB_PATH):
        compile_oracle(_LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get(LIB_ENV) or _LIB_PATH
        if path == _LIB_PATH and not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(path)
        L.or_mix64.restype = ctypes.c_uint64
        L.or_mix64.argtypes = [ctypes.c_uint64]
        L.or_splitmix_nth.restype = ctypes.c_uint64
        L.or_splitmix_nth.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.or_draw_key.restype = ctypes.c_uint64
        L.or_draw_key.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32]
        L.or_below.restype = ctypes.c_uint64
        L.or_below.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.or_floyd.restype = ctypes.c_int
        L.or_floyd.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, I64P]
        L.or_sample_group.restype = ctypes.c_int
        L.or_sample_group.argtypes = [
            ctypes.c_int64, ctypes.c_int64, I64P, I32P, I32P, ctypes.c_int32, ctypes.c_int32,
            ctypes.c_int64, I32P, ctypes.c_int32, ctypes.c_uint64, ctypes.c_int32,
            ctypes.c_int64, I32P, I64P, ctypes.c_int64, I32P, I32P, I64P, I64P]
        L.or_pack_group.restype = ctypes.c_int
        L.or_pack_group.argtypes = [
            ctypes.c_int64, ctypes.c_int64, VP, I32P, ctypes.c_int32, I32P, ctypes.c_int64, I64P,
            ctypes.c_int64, VP, I32P, I64P, I32P, I32P, ctypes.c_int64, I64P]
        L.or_cache_by_frequency.restype = ctypes.c_int
        L.or_cache_by_frequency.argtypes = [ctypes.c_int64, ctypes.c_int32, I32P, ctypes.c_int64,
                                            I64P, ctypes.c_int64, I32P, I32P, I64P]
        L.or_minhash_order.restype = ctypes.c_int
        L.or_minhash_order.argtypes = [ctypes.c_int64, ctypes.c_int32, I32P, ctypes.c_int64, I64P,
                                       I32P, ctypes.c_int64, I32P, ctypes.c_int32, I32P, I32P]
        L.or_assemble_batch.restype = ctypes.c_int
        L.or_assemble_batch.argtypes = [VP, ctypes.c_int64, VP, ctypes.c_int64, I32P,
                                        ctypes.c_int64, ctypes.c_int64, VP]
        _lib = L
    return _lib


def _p(a: np.ndarray, t):
    return a.ctypes.data_as(t)


class OracleError(RuntimeError):
    pass


# ---------------------------------------------------------------- randomness
def mix64(z: int) -> int:
    return lib().or_mix64(z & (2**64 - 1))


def splitmix_nth(state: int, i: int) -> int:
    return lib().or_splitmix_nth(state & (2**64 - 1), i)


def draw_key(rng_seed: int, g: int, k: int, v: int) -> int:
    return lib().or_draw_key(rng_seed & (2**64 - 1), g & (2**64 - 1), k, v)


def below(h: int, m: int) -> int:
    return lib().or_below(h & (2**64 - 1), m)


def floyd(d: int, f: int, key: int) -> list[int]:
    out = np.zeros(max(f, 1), dtype=np.int64)
    rc = lib().or_floyd(d, f, key & (2**64 - 1), _p(out, I64P))
    if rc:
        raise OracleError(f"or_floyd rc={rc}")
    return out[:f].tolist()


# ---------------------------------------------------------------- sampling
def sample_bounds(N: int, E: int, S: int, fanouts, layered=False) -> tuple[int, int]:
    """Per-batch upper bounds on node and edge counts (negative fan-out = all):
    a hop adds at most min(f * frontier, E) edges and as many nodes."""
    n, e, front = S, 0, S
    for f in fanouts:
        hop_e = E if f < 0 else min(front * f, E)
        e += hop_e
        n = min(n + hop_e, N)
        front = n if layered else min(hop_e, N)
    return n, (e if layered else min(e, E))


def host_threads(cap: int = 16) -> int:
    """Host threads for running the oracle on several batches at once: the
    cores this process may run on, at most `cap`."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(cap, n))


def sample_group(offsets, indices, seeds, fanouts, rng_seed, batch_base=0, layered=False,
                 threads=1):
    """Group sampling.  seeds: int32 [B, S].  Returns a dict with per-batch
    numpy arrays: nodes[b], hop_ptr[b], edge_src[b], edge_dst[b], edge_ptr[b].

    threads > 1 runs the (single-threaded) C oracle on runs of consecutive
    batches in that many host threads at once.  Mini-batches are sampled
    independently and each draw is keyed by its global batch number, so the
    result is the same as one call over the whole group."""
    sd = np.ascontiguousarray(seeds, dtype=np.int32)
    B = sd.shape[0]
    threads = max(1, min(int(threads), B))
    if threads > 1:
        from concurrent.futures import ThreadPoolExecutor
        off = np.ascontiguousarray(offsets, dtype=np.int64)
        idx = np.ascontiguousarray(indices, dtype=np.int32)
        cuts = [B * t // threads for t in range(threads + 1)]
        with ThreadPoolExecutor(threads) as ex:  # ctypes calls release the GIL
            parts = list(ex.map(
                lambda t: _sample_one(off, idx, sd[cuts[t]:cuts[t + 1]], fanouts, rng_seed,
                                      batch_base + cuts[t], layered),
                range(threads)))
        out = {k: [x for p in parts for x in p[k]]
               for k in ("nodes", "hop_ptr", "edge_src", "edge_dst", "edge_ptr")}
        out["max_nodes"] = max(p["max_nodes"] for p in parts)
        out["max_edges"] = max(p["max_edges"] for p in parts)
        return out
    return _sample_one(offsets, indices, sd, fanouts, rng_seed, batch_base, layered)


def _sample_one(offsets, indices, seeds, fanouts, rng_seed, batch_base, layered):
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    idx = np.ascontiguousarray(indices, dtype=np.int32)
    sd = np.ascontiguousarray(seeds, dtype=np.int32)
    B, S = sd.shape
    fo = np.ascontiguousarray(fanouts, dtype=np.int32)
    K = len(fo)
    N = len(off) - 1
    E = int(off[-1])
    ncap, ecap = sample_bounds(N, E, S, [int(x) for x in fo], layered)
    ncap, ecap = max(ncap, 1), max(ecap, 1)
    nodes = np.zeros(B * ncap, dtype=np.int32)
    hop = np.zeros(B * (K + 2), dtype=np.int64)
    es = np.zeros(B * ecap, dtype=np.int32)
    ed = np.zeros(B * ecap, dtype=np.int32)
    ep = np.zeros(B * (K + 1), dtype=np.int64)
    need = np.zeros(2, dtype=np.int64)
    rc = lib().or_sample_group(N, E, _p(off, I64P), _p(idx, I32P), _p(sd, I32P), B, S, batch_base,
                               _p(fo, I32P), K, rng_seed & (2**64 - 1), int(layered), ncap,
                               _p(nodes, I32P),
                               _p(hop, I64P), ecap, _p(es, I32P), _p(ed, I32P), _p(ep, I64P),
                               _p(need, I64P))
    if rc:
        raise OracleError(f"or_sample_group rc={rc}")
    hop = hop.reshape(B, K + 2)
    ep = ep.reshape(B, K + 1)
    out = {"nodes": [], "hop_ptr": [], "edge_src": [], "edge_dst": [], "edge_ptr": []}
    for b in range(B):
        n, e = int(hop[b, K + 1]), int(ep[b, K])
        out["nodes"].append(nodes[b * ncap:b * ncap + n].copy())
        out["hop_ptr"].append(hop[b].copy())
        out["edge_src"].append(es[b * ecap:b * ecap + e].copy())
        out["edge_dst"].append(ed[b * ecap:b * ecap + e].copy())
        out["edge_ptr"].append(ep[b].copy())
    out["max_nodes"], out["max_edges"] = int(need[0]), int(need[1])
    return out


# ---------------------------------------------------------------- packing
def pack_group(feats, cache_slot, node_lists, with_unique=True, rows=True, row_bytes=None):
    """Batched packing.  feats: numpy [N, ...] (rows are copied as bytes);
    cache_slot: int32 [N]; node_lists: list of int32 arrays (one per batch).
    rows=False computes the tables only (feats may then be None, with
    row_bytes given)."""
    if rows:
        X = np.ascontiguousarray(feats)
        N = X.shape[0]
        R = X.nbytes // N
    else:
        X = None
        N = len(cache_slot)
        R = row_bytes or 1
    cs = np.ascontiguousarray(cache_slot, dtype=np.int32)
    B = len(node_lists)
    counts = np.array([len(x) for x in node_lists], dtype=np.int64)
    stride = max(int(counts.max()) if B else 0, 1)
    nodes = np.zeros(B * stride, dtype=np.int32)
    for b, x in enumerate(node_lists):
        nodes[b * stride:b * stride + len(x)] = x
    total = int(counts.sum())
    packed = np.zeros((max(total, 1), R), dtype=np.uint8) if rows else None
    pids = np.zeros(max(total, 1), dtype=np.int32)
    pptr = np.zeros(B + 1, dtype=np.int64)
    loc = np.zeros(B * stride, dtype=np.int32)
    uniq = np.zeros(max(total, 1), dtype=np.int32)
    need = np.zeros(3, dtype=np.int64)
    rc = lib().or_pack_group(N, R, X.ctypes.data_as(VP) if rows else None, _p(cs, I32P), B,
                             _p(nodes, I32P), stride, _p(counts, I64P), total,
                             packed.ctypes.data_as(VP) if rows else None, _p(pids, I32P),
                             _p(pptr, I64P), _p(loc, I32P),
                             _p(uniq, I32P) if with_unique else None, total, _p(need, I64P))
    if rc:
        raise OracleError(f"or_pack_group rc={rc}")
    nrows = int(need[0])
    return {
        "packed": packed[:nrows] if rows else None, "packed_ids": pids[:nrows], "packed_ptr": pptr,
        "loc": [loc[b * stride:b * stride + int(counts[b])].copy() for b in range(B)],
        "unique": uniq[:int(need[1])].copy() if with_unique else None,
        "packed_rows": nrows, "unique_nodes": int(need[1]), "unique_packed": int(need[2]),
    }


def assemble_batch(cache, packed_b, loc_b, row_bytes):
    """Feature assembling for one batch: rows from the cache (loc < 0) or the
    batch's packed chunk, in the order of loc_b.  Returns uint8 [n_b, row_bytes]."""
    c = np.ascontiguousarray(cache).view(np.uint8).reshape(-1)
    p = np.ascontiguousarray(packed_b).view(np.uint8).reshape(-1)
    lb = np.ascontiguousarray(loc_b, dtype=np.int32)
    n = len(lb)
    out = np.zeros((n, row_bytes), dtype=np.uint8)
    rc = lib().or_assemble_batch(c.ctypes.data_as(VP), len(c) // row_bytes, p.ctypes.data_as(VP),
                                 len(p) // row_bytes, _p(lb, I32P), n, row_bytes,
                                 out.ctypes.data_as(VP))
    if rc:
        raise OracleError(f"or_assemble_batch rc={rc}")
    return out


def cache_by_frequency(N, node_lists, cache_rows):
    """Access-frequency cache: (cache_slot int32 [N], cache_nodes int32
    [cache_rows] with -1 for empty slots, cached count)."""
    B = len(node_lists)
    counts = np.array([len(x) for x in node_lists], dtype=np.int64)
    stride = max(int(counts.max()) if B else 0, 1)
    nodes = np.zeros(B * stride, dtype=np.int32)
    for b, x in enumerate(node_lists):
        nodes[b * stride:b * stride + len(x)] = x
    slot = np.zeros(N, dtype=np.int32)
    cn = np.zeros(max(cache_rows, 1), dtype=np.int32)
    cached = np.zeros(1, dtype=np.int64)
    rc = lib().or_cache_by_frequency(N, B, _p(nodes, I32P), stride, _p(counts, I64P), cache_rows,
                                     _p(slot, I32P), _p(cn, I32P), _p(cached, I64P))
    if rc:
        raise OracleError(f"or_cache_by_frequency rc={rc}")
    return slot, cn[:cache_rows], int(cached[0])


def minhash_order(N, node_lists, entries, perms):
    """Disk-cache reordering by MinHash (Alg. 1).  perms: int32 [k, B].
    Returns (order int32 [m], signature int32 [m], -1 = in no sample)."""
    B = len(node_lists)
    counts = np.array([len(x) for x in node_lists], dtype=np.int64)
    stride = max(int(counts.max()) if B else 0, 1)
    nodes = np.zeros(B * stride, dtype=np.int32)
    for b, x in enumerate(node_lists):
        nodes[b * stride:b * stride + len(x)] = x
    ent = np.ascontiguousarray(entries, dtype=np.int32)
    pm = np.ascontiguousarray(perms, dtype=np.int32)
    m = len(ent)
    order = np.zeros(max(m, 1), dtype=np.int32)
    sig = np.zeros(max(m, 1), dtype=np.int32)
    rc = lib().or_minhash_order(N, B, _p(nodes, I32P), stride, _p(counts, I64P), _p(ent, I32P),
                                m, _p(pm, I32P), pm.shape[0], _p(order, I32P), _p(sig, I32P))
    if rc:
        raise OracleError(f"or_minhash_order rc={rc}")
    return order[:m], sig[:m]
