// Cache configuration by access frequency (DiskGNN §4 "Four-level hierarchical
// feature store": one counter per node, streamed over the graph samples, and
// the most popular features go to the fastest tier; §3: this placement
// minimises the features fetched from slower storage) and the row gather that
// fills the cache table, which the paper does by treating the cache as a
// special mini-batch of batched packing (§5.2).  The same gather, run once per
// mini-batch over that batch's packed IDs, is the individual packing of §5.2
// (Fig. 6a).
//
// Frequencies: a node's count is the number of mini-batches of the group that
// require it, i.e. the popcount of its membership word.  Ranking (count
// descending, then ID ascending) is a stable counting sort over 65 keys: per
// block counts of every key, a scan down each key's column, then ranks from
// block bases + wave prefixes + ballot prefixes, with no sort.
#include <initializer_list>
#include <string.h>

#include "dg_rows.h"

namespace dg {
namespace {

constexpr int KEYS = 65;           // popcounts 0..64
constexpr int CF_WAVES = 4;
constexpr int CF_THREADS = 64 * CF_WAVES;
constexpr int CF_ROUNDS = 16;
constexpr int CF_BLOCK = 64 * CF_ROUNDS * CF_WAVES;

struct FreqScan {
  const uint64_t *mask;
  uint64_t keep;      // bits of the group's batches
  int64_t N;
  int64_t nblk;
  uint32_t *cnt;      // [nblk][KEYS]
  int64_t *base;      // [nblk][KEYS] exclusive scans down each key
  int64_t *totals;    // [KEYS]
  int64_t first[KEYS];  // rank of the first node of each key (host-computed)
  int64_t cap;          // cache rows
  int32_t *cache_slot;
  int32_t *cache_nodes;
};

__device__ __forceinline__ int key_of(const FreqScan &a, int64_t u) {
  return u < a.N ? __popcll(a.mask[u] & a.keep) : -1;
}

// Counts of every key in one wave tile (lane k < KEYS-1 keeps key k's count;
// key 64 is returned separately).
__device__ __forceinline__ void wave_key_counts(const int (&k)[CF_ROUNDS], int lane,
                                                uint32_t *mine, uint32_t *k64) {
  uint32_t c = 0, top = 0;
#pragma unroll
  for (int r = 0; r < CF_ROUNDS; ++r) {
    int key = k[r];
    uint64_t pending = __ballot(key >= 0);
    while (pending) {  // one iteration per distinct key present in the round
      const int src = __ffsll((long long)pending) - 1;
      const int kk = __shfl(key, src, 64);
      const uint64_t bal = __ballot(key == kk);
      pending &= ~bal;
      if (kk == 64) top += (uint32_t)__popcll(bal);
      else if (lane == kk) c += (uint32_t)__popcll(bal);
    }
  }
  *mine = c;
  *k64 = top;
}

__global__ __launch_bounds__(CF_THREADS) void k_freq_count(FreqScan a) {
  __shared__ uint32_t s_cnt[CF_WAVES][KEYS];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * CF_BLOCK + (int64_t)w * 64 * CF_ROUNDS;
  int k[CF_ROUNDS];
#pragma unroll
  for (int r = 0; r < CF_ROUNDS; ++r) k[r] = key_of(a, t0 + r * 64 + lane);
  uint32_t mine, top;
  wave_key_counts(k, lane, &mine, &top);
  s_cnt[w][lane] = mine;
  if (lane == 0) s_cnt[w][64] = top;
  __syncthreads();
  for (int i = threadIdx.x; i < KEYS; i += CF_THREADS) {
    uint32_t v = 0;
    for (int j = 0; j < CF_WAVES; ++j) v += s_cnt[j][i];
    a.cnt[(size_t)blockIdx.x * KEYS + i] = v;
  }
}

// One block per key: exclusive scan of that key's per-block counts.
__global__ __launch_bounds__(1024) void k_freq_scan(FreqScan a) {
  __shared__ int64_t s_w[16];
  const int key = blockIdx.x;
  int64_t carry = 0;
  for (int64_t c0 = 0; c0 < a.nblk; c0 += 1024) {
    const int64_t i = c0 + threadIdx.x;
    const int64_t v = i < a.nblk ? (int64_t)a.cnt[(size_t)i * KEYS + key] : 0;
    int64_t incl = v;
    for (int o = 1; o < 64; o <<= 1) {
      int64_t y = __shfl_up(incl, o, 64);
      if ((threadIdx.x & 63) >= o) incl += y;
    }
    if ((threadIdx.x & 63) == 63) s_w[threadIdx.x >> 6] = incl;
    __syncthreads();
    int64_t before = 0, sum = 0;
    for (int j = 0; j < 16; ++j) {
      if (j < (int)(threadIdx.x >> 6)) before += s_w[j];
      sum += s_w[j];
    }
    __syncthreads();
    if (i < a.nblk) a.base[(size_t)i * KEYS + key] = carry + before + incl - v;
    carry += sum;
  }
  if (threadIdx.x == 0) a.totals[key] = carry;
}

// Ranks: rank(u) = first[key] + block base + earlier waves + earlier rounds +
// ballot prefix.  Nodes with rank < cap are cached.
__global__ __launch_bounds__(CF_THREADS) void k_freq_place(FreqScan a) {
  __shared__ uint32_t s_cnt[CF_WAVES][KEYS];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * CF_BLOCK + (int64_t)w * 64 * CF_ROUNDS;
  int k[CF_ROUNDS];
#pragma unroll
  for (int r = 0; r < CF_ROUNDS; ++r) k[r] = key_of(a, t0 + r * 64 + lane);
  uint32_t mine, top;
  wave_key_counts(k, lane, &mine, &top);
  s_cnt[w][lane] = mine;
  if (lane == 0) s_cnt[w][64] = top;
  __syncthreads();
  // running rank of key (lane) for lanes 0..63, key 64 kept uniform
  const int64_t *bb = a.base + (size_t)blockIdx.x * KEYS;
  int64_t run = a.first[lane] + bb[lane];
  int64_t run64 = a.first[64] + bb[64];
  for (int j = 0; j < w; ++j) {
    run += s_cnt[j][lane];
    run64 += s_cnt[j][64];
  }
  const uint64_t lt = lanes_below();
#pragma unroll
  for (int r = 0; r < CF_ROUNDS; ++r) {
    const int key = k[r];
    const int64_t u = t0 + r * 64 + lane;
    uint64_t pending = __ballot(key >= 0);
    int64_t rank = -1;
    while (pending) {
      const int src = __ffsll((long long)pending) - 1;
      const int kk = __shfl(key, src, 64);
      const uint64_t bal = __ballot(key == kk);
      pending &= ~bal;
      const int64_t start = kk == 64 ? run64 : read_lane(run, kk);
      if (key == kk) rank = start + __popcll(bal & lt);
      if (kk == 64) run64 += __popcll(bal);
      else if (lane == kk) run += __popcll(bal);
    }
    if (key >= 0) {
      const bool cached = key > 0 && rank < a.cap;
      a.cache_slot[u] = cached ? (int32_t)rank : -1;
      if (cached) a.cache_nodes[rank] = (int32_t)u;
    }
  }
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// ------------------------------------------------------------------ row gather
constexpr int G_THREADS = 256;
constexpr int G_UNROLL = 4;

template <int LPR, int CPL>
__global__ __launch_bounds__(G_THREADS) void k_gather16(const v4u *X, int64_t N,
                                                        const int32_t *ids, int64_t n, int C,
                                                        v4u *out, uint32_t *err) {
  constexpr int GPB = G_THREADS / LPR;
  const int sub = threadIdx.x % LPR;
  const int64_t grp = (int64_t)blockIdx.x * GPB + threadIdx.x / LPR;
  const int64_t ngrp = (int64_t)gridDim.x * GPB;
  for (int64_t j0 = grp * G_UNROLL; j0 < n; j0 += ngrp * G_UNROLL) {
    const v4u *src[G_UNROLL];
#pragma unroll
    for (int u = 0; u < G_UNROLL; ++u) {
      const int64_t j = j0 + u;
      src[u] = nullptr;
      if (j < n) {
        const int32_t id = ids[j];
        if (id >= 0 && (int64_t)id < N) src[u] = X + (int64_t)id * C;
        else if (sub == 0 && err) atomicOr(err, ERR_NODE_RANGE);
      }
    }
    v4u v[G_UNROLL][CPL];
#pragma unroll
    for (int u = 0; u < G_UNROLL; ++u)
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int ch = sub + c * LPR;
        v[u][c] = (src[u] && ch < C) ? ld_stream(src[u] + ch) : v4u{0u, 0u, 0u, 0u};
      }
#pragma unroll
    for (int u = 0; u < G_UNROLL; ++u) {
      const int64_t j = j0 + u;
      if (j < n) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const int ch = sub + c * LPR;
          if (ch < C) st_stream(v[u][c], out + j * C + ch);
        }
      }
    }
  }
}

template <typename T>
__global__ __launch_bounds__(G_THREADS) void k_gather_any(const T *X, int64_t N, const int32_t *ids,
                                                          int64_t n, int64_t W, T *out,
                                                          uint32_t *err) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * G_THREADS + threadIdx.x) >> 6;
  const int64_t nwave = ((int64_t)gridDim.x * G_THREADS) >> 6;
  for (int64_t j = wave; j < n; j += nwave) {
    const int32_t id = ids[j];
    const bool ok = id >= 0 && (int64_t)id < N;
    if (!ok && lane == 0 && err) atomicOr(err, ERR_NODE_RANGE);
    for (int64_t c = lane; c < W; c += 64)
      out[j * W + c] = ok ? X[(int64_t)id * W + c] : zero_word<T>();
  }
}

template <int LPR, int CPL>
void gather16(const void *X, int64_t N, const int32_t *ids, int64_t n, int C, void *out,
              uint32_t *err, hipStream_t s) {
  constexpr int GPB = G_THREADS / LPR;
  int64_t blocks = ((n + G_UNROLL - 1) / G_UNROLL + GPB - 1) / GPB;
  if (blocks > (1ll << 20)) blocks = 1ll << 20;
  hipLaunchKernelGGL((k_gather16<LPR, CPL>), dim3((unsigned)blocks), dim3(G_THREADS), 0, s,
                     (const v4u *)X, N, ids, n, C, (v4u *)out, err);
}

template <typename T>
void gather_any(const void *X, int64_t N, const int32_t *ids, int64_t n, int64_t row_bytes,
                void *out, uint32_t *err, hipStream_t s) {
  int64_t blocks = (n + 3) / 4;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_gather_any<T>, dim3((unsigned)blocks), dim3(G_THREADS), 0, s,
                     (const T *)X, N, ids, n, row_bytes / (int64_t)sizeof(T), (T *)out, err);
}

bool overlaps(const void *a, int64_t an, const void *b, int64_t bn) {
  if (!a || !b || an <= 0 || bn <= 0) return false;
  uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + (uintptr_t)bn && y < x + (uintptr_t)an;
}

}  // namespace

int launch_gather(const void *X, int64_t N, int64_t row_bytes, const int32_t *ids, int64_t n,
                  void *out, uint32_t *err, hipStream_t s) {
  if (n == 0) return DG_OK;
  const int w = word_bytes(row_bytes, {X, out});
  RowShape sh;
  if (w == 16 && row_shape16(row_bytes / 16, &sh)) {
    const int C = (int)(row_bytes / 16);
    if (sh.lpr == 4) gather16<4, 1>(X, N, ids, n, C, out, err, s);
    else if (sh.lpr == 8) gather16<8, 1>(X, N, ids, n, C, out, err, s);
    else if (sh.lpr == 16) gather16<16, 1>(X, N, ids, n, C, out, err, s);
    else if (sh.lpr == 32 && sh.cpl == 1) gather16<32, 1>(X, N, ids, n, C, out, err, s);
    else if (sh.lpr == 64 && sh.cpl == 1) gather16<64, 1>(X, N, ids, n, C, out, err, s);
    else if (sh.lpr == 32 && sh.cpl == 3) gather16<32, 3>(X, N, ids, n, C, out, err, s);
    else if (sh.lpr == 64 && sh.cpl == 2) gather16<64, 2>(X, N, ids, n, C, out, err, s);
    else gather16<64, 4>(X, N, ids, n, C, out, err, s);
  } else if (w == 16) {
    gather_any<uint4>(X, N, ids, n, row_bytes, out, err, s);
  } else if (w == 8) {
    gather_any<uint2>(X, N, ids, n, row_bytes, out, err, s);
  } else if (w == 4) {
    gather_any<uint32_t>(X, N, ids, n, row_bytes, out, err, s);
  } else if (w == 2) {
    gather_any<uint16_t>(X, N, ids, n, row_bytes, out, err, s);
  } else {
    gather_any<uint8_t>(X, N, ids, n, row_bytes, out, err, s);
  }
  DG_HIP(hipGetLastError());
  return DG_OK;
}

}  // namespace dg

using namespace dg;

extern "C" size_t dg_cache_workspace_bytes(int64_t num_nodes) {
  if (num_nodes < 1) return 0;
  const int64_t nblk = (num_nodes + CF_BLOCK - 1) / CF_BLOCK;
  Carve c(nullptr);
  (void)c.take<uint32_t>((size_t)nblk * KEYS);
  (void)c.take<int64_t>((size_t)nblk * KEYS);
  (void)c.take<int64_t>(KEYS);
  return c.used;
}

extern "C" int dg_cache_by_frequency(const uint64_t *membership, int64_t N, int32_t B,
                                     int64_t cache_rows, int32_t *cache_slot,
                                     int32_t *cache_nodes, int64_t *cached, void *ws,
                                     size_t ws_bytes, hipStream_t stream) {
  if (!membership || !cache_slot || !cached || (cache_rows > 0 && !cache_nodes))
    return set_error(DG_EINVAL, "dg_cache_by_frequency: null pointer argument");
  if (N < 1 || N > 0x7fffffffll || B < 1 || B > DG_MAX_BATCHES || cache_rows < 0 ||
      cache_rows > N)
    return set_error(DG_EINVAL, "dg_cache_by_frequency: bad sizes");
  const size_t need = dg_cache_workspace_bytes(N);
  if (!ws || ws_bytes < need || ((uintptr_t)ws & 255))
    return set_error(DG_EWORKSPACE, "dg_cache_by_frequency: workspace needs %zu bytes", need);
  hipStream_t s = stream;
  FreqScan a;
  memset(&a, 0, sizeof(a));
  a.mask = membership;
  a.keep = B == 64 ? ~0ull : ((1ull << B) - 1ull);
  a.N = N;
  a.nblk = (N + CF_BLOCK - 1) / CF_BLOCK;
  Carve c(ws);
  a.cnt = c.take<uint32_t>((size_t)a.nblk * KEYS);
  a.base = c.take<int64_t>((size_t)a.nblk * KEYS);
  a.totals = c.take<int64_t>(KEYS);
  a.cap = cache_rows;
  a.cache_slot = cache_slot;
  a.cache_nodes = cache_nodes;
  hipLaunchKernelGGL(k_freq_count, dim3((unsigned)a.nblk), dim3(CF_THREADS), 0, s, a);
  hipLaunchKernelGGL(k_freq_scan, dim3(KEYS), dim3(1024), 0, s, a);
  DG_HIP(hipGetLastError());
  int64_t totals[KEYS];
  DG_HIP(hipMemcpyAsync(totals, a.totals, sizeof(totals), hipMemcpyDeviceToHost, s));
  DG_HIP(hipStreamSynchronize(s));
  // keys in rank order: 64, 63, ..., 1, then 0 (never cached)
  int64_t run = 0;
  for (int k = 64; k >= 1; --k) {
    a.first[k] = run;
    run += totals[k];
  }
  a.first[0] = run;
  const int64_t accessed = run;
  *cached = accessed < cache_rows ? accessed : cache_rows;
  if (cache_rows > 0)
    hipLaunchKernelGGL(k_fill_i32, dim3(256), dim3(256), 0, s, cache_nodes, cache_rows, -1);
  hipLaunchKernelGGL(k_freq_place, dim3((unsigned)a.nblk), dim3(CF_THREADS), 0, s, a);
  DG_HIP(hipGetLastError());
  DG_HIP(hipStreamSynchronize(s));
  return DG_OK;
}

extern "C" int dg_gather_rows(const void *feats, int64_t N, int64_t row_bytes,
                              const int32_t *ids, int64_t n, void *out, int32_t *status,
                              hipStream_t stream) {
  if (n < 0 || row_bytes < 1 || N < 1)
    return set_error(DG_EINVAL, "dg_gather_rows: bad sizes");
  if (n == 0) return DG_OK;
  if (!feats || !ids || !out) return set_error(DG_EINVAL, "dg_gather_rows: null pointer argument");
  if (overlaps(out, n * row_bytes, feats, N * row_bytes) || overlaps(out, n * row_bytes, ids, n * 4))
    return set_error(DG_EINVAL, "dg_gather_rows: output overlaps an input");
  return launch_gather(feats, N, row_bytes, ids, n, out, reinterpret_cast<uint32_t *>(status),
                       stream);
}
