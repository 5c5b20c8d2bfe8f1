"""Seeded synthetic inputs for the offline-sampling path.

This package holds input generators only — graphs, feature tables, seed
batches and cache sets — and none of the method's arithmetic (no sampling, no
deduplication, no packing).  Both the device path and the CPU oracle take their
inputs from here.  Every draw is counter-based (a hash of a purpose stream and
an element counter), so results do not depend on thread count or chunking, and
the integer parts (graphs, seeds, cache sets) are identical on CPU and GPU.
Feature values come from torch's normal generator on the device they are made
on; they are opaque bytes to the path.

Workloads (the paper's datasets are not available; these stand in for them —
Table 2 shapes: Ogbn-papers100M ~ 111M nodes with 128-d fp32 features,
Friendster ~ 66M nodes; sampling setting of §7.1: node-wise, fan-outs over 3
hops, 1024 seeds per mini-batch):

  T     10,000-node random directed graph, out-degree ~ U{1..20}, targets
        uniform and distinct, fp32 dim 16, fan-out [5,5], 4 x 64 seeds, cache
        = top 10% by in-degree.
  M1    R-MAT (0.57,0.19,0.19,0.05), 1M nodes, 16M draws, fp32 dim 128,
        fan-out [15,10,5], 32 x 1024 seeds, cache 10%.
  L100  R-MAT default, 100M nodes, 1.6B draws, fp32 dim 128 (51.2 GB),
        fan-out [15,10,5], 64 x 1024 seeds, cache 5%.
  W120  R-MAT default, 120M nodes, 1.7B draws, fp16 dim 768 (184 GB),
        fan-out [25,15], 64 x 1024 seeds, cache 2%.
  H65   R-MAT (0.6,0.15,0.15,0.1), 65M nodes, 1.8B draws, fp32 dim 256,
        fan-out [20,15,10], 16 x 4096 seeds, cache {0,10,30}%.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

MASK64 = (1 << 64) - 1

# purpose streams derived from the workload seed
STREAM_GRAPH = 1
STREAM_RELABEL = 2
STREAM_SEEDS = 3
STREAM_FEATS = 4
STREAM_SAMPLER = 5


def _s64(c: int) -> int:
    """Unsigned 64-bit constant as the equal-bits signed value torch stores."""
    c &= MASK64
    return c - (1 << 64) if c >= (1 << 63) else c


_M1 = _s64(0xFF51AFD7ED558CCD)
_M2 = _s64(0xC4CEB9FE1A85EC53)
_INC = _s64(0xD1B54A32D192ED03)


def _lsr(x: torch.Tensor, s: int) -> torch.Tensor:
    return (x >> s) & ((1 << (64 - s)) - 1)


def fmix64(x: torch.Tensor) -> torch.Tensor:
    """MurmurHash3's 64-bit finaliser on int64 tensors (wrapping arithmetic)."""
    x = x ^ _lsr(x, 33)
    x = x * _M1
    x = x ^ _lsr(x, 33)
    x = x * _M2
    return x ^ _lsr(x, 33)


def _fmix64_int(x: int) -> int:
    x &= MASK64
    x ^= x >> 33
    x = (x * 0xFF51AFD7ED558CCD) & MASK64
    x ^= x >> 33
    x = (x * 0xC4CEB9FE1A85EC53) & MASK64
    return x ^ (x >> 33)


def stream_key(seed: int, stream: int) -> int:
    """64-bit key of one purpose stream of a workload seed."""
    return _fmix64_int(_fmix64_int(seed) ^ (stream * 0x632BE59BD9B4E019))


def hash_u32(key: int, counter: torch.Tensor) -> torch.Tensor:
    """Uniform 32-bit values (as int64 in [0, 2^32)) for each counter."""
    return _lsr(fmix64(counter * _INC + _s64(key)), 32)


def sampler_seed(seed: int) -> int:
    """The rng_seed handed to the sampler for a workload seed."""
    return stream_key(seed, STREAM_SAMPLER)


# --------------------------------------------------------------- permutations
def feistel_permute(x: torch.Tensor, n: int, key: int, rounds: int = 4) -> torch.Tensor:
    """Keyed bijection of [0, n) (balanced Feistel network over an even number
    of bits, with cycle walking back into [0, n)).  x: int64 values in [0, n)."""
    bits = max(2, math.ceil(math.log2(max(n, 2))))
    bits += bits & 1
    half = bits // 2
    hmask = (1 << half) - 1

    def enc(y):
        L = y >> half
        R = y & hmask
        for r in range(rounds):
            F = hash_u32(stream_key(key, 100 + r), R) & hmask
            L, R = R, L ^ F
        return (L << half) | R

    y = enc(x)
    walk = torch.nonzero(y >= n).squeeze(1)
    while walk.numel():  # cycle walking: re-encrypt only the values still outside
        z = enc(y[walk])
        y[walk] = z
        walk = walk[z >= n]
    return y


# --------------------------------------------------------------- graphs
def uniform_graph(n: int, dmin: int, dmax: int, seed: int):
    """Directed graph: each node gets U{dmin..dmax} out-neighbours, drawn
    uniformly among the other nodes, distinct; rows sorted.  CPU, numpy.
    Returns (offsets int64 [n+1], indices int32 [E])."""
    key = stream_key(seed, STREAM_GRAPH)
    v = torch.arange(n, dtype=torch.int64)
    span = dmax - dmin + 1
    deg = (dmin + ((hash_u32(key, v * 4096) * span) >> 32)).numpy()
    tries = 4 * dmax + 16
    ctr = v[:, None] * 4096 + 1 + torch.arange(tries, dtype=torch.int64)[None, :]
    t = (hash_u32(key, ctr) * (n - 1)) >> 32
    t = (t + (t >= v[:, None]).long()).numpy()  # skip the node itself
    rows = []
    for u in range(n):
        d = int(deg[u])
        chosen: list[int] = []
        for x in t[u]:  # first d distinct draws, in draw order
            if len(chosen) == d:
                break
            if int(x) not in chosen:
                chosen.append(int(x))
        if len(chosen) < d:
            raise RuntimeError("uniform_graph: too many repeated draws")
        rows.append(sorted(chosen))
    offsets = np.zeros(n + 1, dtype=np.int64)
    offsets[1:] = np.cumsum([len(r) for r in rows])
    indices = np.fromiter((x for r in rows for x in r), dtype=np.int32, count=int(offsets[-1]))
    return offsets, indices


def rmat_edges(n: int, draws: int, a: float, b: float, c: float, seed: int,
               device="cpu", chunk: int = 1 << 26) -> torch.Tensor:
    """R-MAT edge draws (Chakrabarti, Zhan & Faloutsos, SDM 2004) at scale
    ceil(log2 n); each level's quadrant comes from a 16-bit slice of a 64-bit
    counter hash (four levels per hash); a draw with an endpoint >= n is
    redrawn.  Endpoints are then relabelled by a keyed permutation (hubs
    scattered over the ID range).  Returns int64 keys src*n + dst of the
    distinct non-loop edges, ascending."""
    scale = max(1, math.ceil(math.log2(n)))
    key = stream_key(seed, STREAM_GRAPH)
    rkey = stream_key(seed, STREAM_RELABEL)
    ta, tb, tc = (int(round(p * 2**16)) for p in (a, a + b, a + b + c))
    keys = []
    for start in range(0, draws, chunk):
        m = min(chunk, draws - start)
        e = torch.arange(start, start + m, dtype=torch.int64, device=device)
        src = torch.zeros(m, dtype=torch.int64, device=device)
        dst = torch.zeros(m, dtype=torch.int64, device=device)
        todo = torch.arange(m, dtype=torch.int64, device=device)
        for attempt in range(64):
            ee = e[todo]
            s = torch.zeros_like(ee)
            d = torch.zeros_like(ee)
            for lvl in range(scale):
                if lvl % 4 == 0:
                    h = fmix64(((ee << 9) | ((lvl // 4) << 6) | attempt) * _INC + _s64(key))
                r = (h >> (16 * (lvl % 4))) & 0xFFFF
                s = (s << 1) | (r >= tb).long()
                d = (d << 1) | (((r >= ta) & (r < tb)) | (r >= tc)).long()
            src[todo] = s
            dst[todo] = d
            bad = (s >= n) | (d >= n)
            todo = todo[bad]
            if todo.numel() == 0:
                break
        if todo.numel():
            raise RuntimeError("R-MAT rejection did not converge")
        src = feistel_permute(src, n, rkey)
        dst = feistel_permute(dst, n, rkey)
        keep = src != dst
        keys.append(src[keep] * n + dst[keep])
        del src, dst, e
    allk = torch.cat(keys)
    del keys
    return torch.unique(allk, sorted=True)


def csr_from_keys(keys: torch.Tensor, n: int):
    """CSR (offsets int64 [n+1], indices int32) from ascending src*n+dst keys."""
    src = keys // n
    counts = torch.bincount(src, minlength=n)
    del src
    offsets = torch.zeros(n + 1, dtype=torch.int64, device=keys.device)
    offsets[1:] = torch.cumsum(counts, 0)
    indices = (keys % n).to(torch.int32)
    return offsets, indices


def rmat_graph(n, draws, a, b, c, seed, device="cpu"):
    keys = rmat_edges(n, draws, a, b, c, seed, device)
    g = csr_from_keys(keys, n)
    del keys
    return g


# --------------------------------------------------------------- other inputs
def seed_batches(n: int, B: int, S: int, seed: int, device="cpu", offsets=None) -> torch.Tensor:
    """B x S seed nodes drawn without replacement: a keyed permutation of
    [0, n) is walked in order and the first B*S nodes with at least one
    out-neighbour are kept (seeds are training nodes, which in the paper's
    datasets sit in the graph's connected part); they are split consecutively
    into batches.  Without `offsets` every node is eligible."""
    key = stream_key(seed, STREAM_SEEDS)
    need = B * S
    if offsets is None:
        if need > n:
            raise ValueError("more seeds than nodes")
        i = torch.arange(need, dtype=torch.int64, device=device)
        return feistel_permute(i, n, key).to(torch.int32).reshape(B, S)
    deg = offsets[1:] - offsets[:-1]
    out, have, start = [], 0, 0
    step = max(4 * need, 1 << 16)
    while have < need:
        if start >= n:
            raise ValueError("fewer nodes with out-neighbours than seeds")
        i = torch.arange(start, min(n, start + step), dtype=torch.int64, device=device)
        v = feistel_permute(i, n, key)
        v = v[deg[v] > 0]
        out.append(v[:need - have])
        have += out[-1].numel()
        start += step
    return torch.cat(out).to(torch.int32).reshape(B, S)


def features(n: int, dim: int, dtype, seed: int, device="cpu", chunk_rows: int = 1 << 22):
    """Feature table [n, dim] ~ N(0,1) (fp16 tables: fp32 draws rounded to
    nearest even)."""
    gen = torch.Generator(device=device)
    gen.manual_seed(stream_key(seed, STREAM_FEATS) & ((1 << 63) - 1))
    X = torch.empty((n, dim), dtype=dtype, device=device)
    for r0 in range(0, n, chunk_rows):
        r1 = min(n, r0 + chunk_rows)
        if dtype == torch.float32:
            X[r0:r1] = torch.randn((r1 - r0, dim), generator=gen, device=device)
        else:
            X[r0:r1] = torch.randn((r1 - r0, dim), generator=gen, device=device,
                                   dtype=torch.float32).to(dtype)
    return X


def cache_by_indegree(indices: torch.Tensor, n: int, count: int):
    """Cache set: the `count` nodes of highest in-degree (ties: lower ID first).
    Returns (cache_slot int32 [n], -1 = not cached, slot = rank; cache_nodes
    int64 [count])."""
    indeg = torch.bincount(indices.to(torch.int64), minlength=n)
    order = torch.sort(indeg, descending=True, stable=True).indices
    cache_nodes = order[:count].clone()
    del order, indeg
    slot = torch.full((n,), -1, dtype=torch.int32, device=indices.device)
    slot[cache_nodes] = torch.arange(count, dtype=torch.int32, device=indices.device)
    return slot, cache_nodes


# --------------------------------------------------------------- workloads
@dataclass
class Config:
    name: str
    n: int
    graph: str                 # "uniform" or "rmat"
    draws: int                 # R-MAT draws (nominal edges)
    abc: tuple = (0.57, 0.19, 0.19)
    dim: int = 128
    dtype: torch.dtype = torch.float32
    fanouts: tuple = (15, 10, 5)
    B: int = 32
    S: int = 1024
    cache_pct: tuple = (10,)   # cache size(s) in percent of n
    seed: int = 0
    degree_range: tuple = (1, 20)

    @property
    def row_bytes(self) -> int:
        return self.dim * torch.tensor([], dtype=self.dtype).element_size()


CONFIGS = {
    "T": Config("T", 10_000, "uniform", 0, dim=16, fanouts=(5, 5), B=4, S=64, cache_pct=(10,)),
    "M1": Config("M1", 1_000_000, "rmat", 16_000_000, fanouts=(15, 10, 5), B=32, S=1024,
                 cache_pct=(10,)),
    "L100": Config("L100", 100_000_000, "rmat", 1_600_000_000, fanouts=(15, 10, 5), B=64,
                   S=1024, cache_pct=(5,)),
    "W120": Config("W120", 120_000_000, "rmat", 1_700_000_000, dim=768, dtype=torch.float16,
                   fanouts=(25, 15), B=64, S=1024, cache_pct=(2,)),
    "H65": Config("H65", 65_000_000, "rmat", 1_800_000_000, abc=(0.6, 0.15, 0.15), dim=256,
                  fanouts=(20, 15, 10), B=16, S=4096, cache_pct=(0, 10, 30)),
}


@dataclass
class Workload:
    cfg: Config
    offsets: torch.Tensor
    indices: torch.Tensor
    seeds: torch.Tensor
    feats: torch.Tensor | None = None
    cache_slot: torch.Tensor | None = None
    cache_nodes: torch.Tensor | None = None
    cache: torch.Tensor | None = None
    rng_seed: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return self.cfg.n

    @property
    def num_edges(self) -> int:
        return int(self.offsets[-1])


def make_graph(cfg: Config, device="cpu"):
    if cfg.graph == "uniform":
        off, idx = uniform_graph(cfg.n, cfg.degree_range[0], cfg.degree_range[1], cfg.seed)
        return torch.from_numpy(off).to(device), torch.from_numpy(idx).to(device)
    a, b, c = cfg.abc
    return rmat_graph(cfg.n, cfg.draws, a, b, c, cfg.seed, device)


def set_cache(w: Workload, pct: int):
    """(Re)build the cache set and cache table for `pct` percent of the nodes."""
    count = w.cfg.n * pct // 100
    w.cache = None
    w.cache_slot, w.cache_nodes = cache_by_indegree(w.indices, w.cfg.n, count)
    if w.feats is not None:
        w.cache = w.feats.index_select(0, w.cache_nodes)
    return w


def make_workload(name_or_cfg, device="cpu", feats=True, cache_pct=None, feats_device=None):
    """Build a whole workload.  Integer inputs are made on `device`; the feature
    table on `feats_device` (default: `device`)."""
    cfg = CONFIGS[name_or_cfg] if isinstance(name_or_cfg, str) else name_or_cfg
    off, idx = make_graph(cfg, device)
    if torch.device(device).type == "cuda":
        torch.cuda.empty_cache()  # give generation temporaries back before the feature table
    seeds = seed_batches(cfg.n, cfg.B, cfg.S, cfg.seed, device, offsets=off)
    w = Workload(cfg, off, idx, seeds, rng_seed=sampler_seed(cfg.seed))
    if feats:
        fd = feats_device or device
        w.feats = features(cfg.n, cfg.dim, cfg.dtype, cfg.seed, fd)
        if str(fd) != str(device):
            w.feats = w.feats.to(device)
    set_cache(w, cfg.cache_pct[0] if cache_pct is None else cache_pct)
    return w
