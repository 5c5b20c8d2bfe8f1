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
// descending, then ID ascending) is a stable counting sort over 65 keys.
//
// The same counting sort orders the disk-cache entries by MinHash value
// (§5.1, Alg. 1): with k hash functions H_j (permutations of the sample IDs,
// given as input), S(v) is the minimum of H_j(i) over every hash function j
// and every sample i that requires v, which equals the minimum over those
// samples of M(i) = min_j H_j(i); entries are then sorted by S.
#include <initializer_list>
#include <string.h>

#include "dg_rows.h"

namespace dg {
namespace {

constexpr int KEYS = 65;  // keys 0..64
constexpr int CF_WAVES = 4;
constexpr int CF_THREADS = 64 * CF_WAVES;
constexpr int CF_ROUNDS = 16;
constexpr int CF_BLOCK = 64 * CF_ROUNDS * CF_WAVES;

// A stable counting sort of a list by a key in 0..64: per-block counts of
// every key, a scan down each key's column, then ranks from block bases +
// earlier waves + earlier rounds + ballot prefixes.  Two uses:
//   FREQ:    list = nodes 0..N-1, key = access count (popcount of the
//            membership word), ranked by count descending;
//   MINHASH: list = the disk-cache entries V_d, key = the entry's MinHash
//            value (64 = in no sample), ranked ascending.
enum Mode { FREQ = 0, MINHASH = 1 };

struct KeySort {
  const uint64_t *mask;
  uint64_t keep;      // bits of the group's batches
  int64_t N;          // nodes
  int64_t n;          // list length
  int64_t nblk;
  uint32_t *cnt;      // [nblk][KEYS]
  int64_t *base;      // [nblk][KEYS] exclusive scans down each key
  int64_t *totals;    // [KEYS]
  int64_t first[KEYS];  // rank of the first element of each key (host-computed)
  uint32_t *err;
  // FREQ outputs
  int64_t cap;
  int32_t *cache_slot;
  int32_t *cache_nodes;
  // MINHASH input / outputs
  const int32_t *ids;    // V_d
  const int32_t *minv;   // [64] min over hash functions of each sample's value
  int32_t *order;        // V_r
  int32_t *signature;    // S(v) per entry (-1: in no sample)
};

template <int MODE>
__device__ __forceinline__ int key_of(const KeySort &a, int64_t i, const int32_t *s_minv) {
  if (i >= a.n) return -1;
  if (MODE == FREQ) return __popcll(a.mask[i] & a.keep);
  const int32_t v = a.ids[i];
  if (v < 0 || (int64_t)v >= a.N) {
    atomicOr(a.err, ERR_NODE_RANGE);
    return 64;
  }
  uint64_t m = a.mask[v] & a.keep;
  int key = 64;  // S(v) = inf: v is required by no sample
  while (m) {
    const int b = __ffsll((long long)m) - 1;
    m &= m - 1;
    key = min(key, s_minv[b]);
  }
  return key;
}

template <int MODE>
__device__ __forceinline__ void load_keys(const KeySort &a, int64_t t0, int lane,
                                          const int32_t *s_minv, int (&k)[CF_ROUNDS]) {
#pragma unroll
  for (int r = 0; r < CF_ROUNDS; ++r) k[r] = key_of<MODE>(a, t0 + r * 64 + lane, s_minv);
}

// Counts of every key in one wave tile (lane k < 64 keeps key k's count; key 64
// is returned separately).
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

template <int MODE>
__device__ __forceinline__ void stage_minv(const KeySort &a, int32_t *s_minv) {
  if (MODE == MINHASH && threadIdx.x < 64) s_minv[threadIdx.x] = a.minv[threadIdx.x];
  __syncthreads();
}

template <int MODE>
__global__ __launch_bounds__(CF_THREADS) void k_key_count(KeySort a) {
  __shared__ uint32_t s_cnt[CF_WAVES][KEYS];
  __shared__ int32_t s_minv[64];
  stage_minv<MODE>(a, s_minv);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * CF_BLOCK + (int64_t)w * 64 * CF_ROUNDS;
  int k[CF_ROUNDS];
  load_keys<MODE>(a, t0, lane, s_minv, k);
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
__global__ __launch_bounds__(1024) void k_key_scan(KeySort a) {
  __shared__ int64_t s_w[16];
  const int key = blockIdx.x;
  int64_t carry = 0;
  for (int64_t c0 = 0; c0 < a.nblk; c0 += 1024) {
    const int64_t i = c0 + threadIdx.x;
    const int64_t v = i < a.nblk ? (int64_t)a.cnt[(size_t)i * KEYS + key] : 0;
    int64_t incl = wave_incl_sum(v);
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

template <int MODE>
__global__ __launch_bounds__(CF_THREADS) void k_key_place(KeySort a) {
  __shared__ uint32_t s_cnt[CF_WAVES][KEYS];
  __shared__ int32_t s_minv[64];
  stage_minv<MODE>(a, s_minv);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * CF_BLOCK + (int64_t)w * 64 * CF_ROUNDS;
  int k[CF_ROUNDS];
  load_keys<MODE>(a, t0, lane, s_minv, k);
  uint32_t mine, top;
  wave_key_counts(k, lane, &mine, &top);
  s_cnt[w][lane] = mine;
  if (lane == 0) s_cnt[w][64] = top;
  __syncthreads();
  const int64_t *bb = a.base + (size_t)blockIdx.x * KEYS;
  int64_t run = a.first[lane] + bb[lane];  // running rank of key `lane`
  int64_t run64 = a.first[64] + bb[64];
  for (int j = 0; j < w; ++j) {
    run += s_cnt[j][lane];
    run64 += s_cnt[j][64];
  }
  const uint64_t lt = lanes_below();
#pragma unroll
  for (int r = 0; r < CF_ROUNDS; ++r) {
    const int key = k[r];
    const int64_t i = t0 + r * 64 + lane;
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
      if (MODE == FREQ) {
        const bool cached = key > 0 && rank < a.cap;
        a.cache_slot[i] = cached ? (int32_t)rank : -1;
        if (cached) a.cache_nodes[rank] = (int32_t)i;
      } else {
        a.order[rank] = a.ids[i];
        if (a.signature) a.signature[i] = key == 64 ? -1 : key;
      }
    }
  }
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// M(i) = min over the k hash functions of H_j(i); values checked to lie in [0, B).
__global__ void k_minhash_min(const int32_t *perms, int32_t k, int32_t B, int32_t *minv,
                              uint32_t *err) {
  const int i = threadIdx.x;
  if (i >= 64) return;
  int32_t m = 64;
  if (i < B) {
    for (int j = 0; j < k; ++j) {
      const int32_t h = perms[(int64_t)j * B + i];
      if (h < 0 || h >= B) atomicOr(err, ERR_ROW_RANGE);
      else m = min(m, h);
    }
  }
  minv[i] = m;
}

int64_t key_blocks(int64_t n) { return (n + CF_BLOCK - 1) / CF_BLOCK; }

void carve_keysort(KeySort &a, Carve &c) {
  a.nblk = key_blocks(a.n);
  a.cnt = c.take<uint32_t>((size_t)a.nblk * KEYS);
  a.base = c.take<int64_t>((size_t)a.nblk * KEYS);
  a.totals = c.take<int64_t>(KEYS);
}

// count pass + scans; returns the per-key totals on the host.
template <int MODE>
int keysort_count(KeySort &a, int64_t *totals, hipStream_t s) {
  if (a.nblk == 0) {
    for (int k = 0; k < KEYS; ++k) totals[k] = 0;
    return DG_OK;
  }
  hipLaunchKernelGGL(k_key_count<MODE>, dim3((unsigned)a.nblk), dim3(CF_THREADS), 0, s, a);
  hipLaunchKernelGGL(k_key_scan, dim3(KEYS), dim3(1024), 0, s, a);
  DG_HIP(hipGetLastError());
  DG_TRY(read_to_host(totals, a.totals, sizeof(int64_t) * KEYS, s));
  return DG_OK;
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
    // Unconditional loads at always-valid addresses, as in the assembly
    // kernel: ids of positions past n are read at n - 1, an id outside [0, N)
    // reads the output row it would write (its row is written as zeros and
    // the error flag set), and a lane past the row reads the row's last vector.
    int32_t id[G_UNROLL];
#pragma unroll
    for (int u = 0; u < G_UNROLL; ++u) id[u] = ids[j0 + u < n ? j0 + u : n - 1];
    const v4u *src[G_UNROLL];
    bool ok[G_UNROLL];
    bool bad = false;
#pragma unroll
    for (int u = 0; u < G_UNROLL; ++u) {
      const int64_t j = j0 + u < n ? j0 + u : n - 1;
      ok[u] = id[u] >= 0 && (int64_t)id[u] < N;
      bad |= j0 + u < n && !ok[u];
      src[u] = ok[u] ? X + (int64_t)id[u] * C : out + j * C;
    }
    v4u v[G_UNROLL][CPL];
#pragma unroll
    for (int u = 0; u < G_UNROLL; ++u)
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int ch = sub + c * LPR;
        v[u][c] = ld_stream(src[u] + (ch < C ? ch : C - 1));
      }
    if (bad && sub == 0 && err) atomicOr(err, ERR_NODE_RANGE);
#pragma unroll
    for (int u = 0; u < G_UNROLL; ++u) {
      const int64_t j = j0 + u;
      if (j < n) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const int ch = sub + c * LPR;
          if (ch < C) st_stream(ok[u] ? v[u][c] : v4u{0u, 0u, 0u, 0u}, out + j * C + ch);
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
  KeySort a;
  memset(&a, 0, sizeof(a));
  a.n = num_nodes;
  Carve c(nullptr);
  carve_keysort(a, c);
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
  KeySort a;
  memset(&a, 0, sizeof(a));
  a.mask = membership;
  a.keep = B == 64 ? ~0ull : ((1ull << B) - 1ull);
  a.N = N;
  a.n = N;
  Carve c(ws);
  carve_keysort(a, c);
  a.cap = cache_rows;
  a.cache_slot = cache_slot;
  a.cache_nodes = cache_nodes;
  int64_t totals[KEYS];
  int rc;
  if ((rc = keysort_count<FREQ>(a, totals, s))) return rc;
  // keys in rank order: 64, 63, ..., 1, then 0 (never cached)
  int64_t run = 0;
  for (int k = 64; k >= 1; --k) {
    a.first[k] = run;
    run += totals[k];
  }
  a.first[0] = run;
  *cached = run < cache_rows ? run : cache_rows;
  if (cache_rows > 0)
    hipLaunchKernelGGL(k_fill_i32, dim3(256), dim3(256), 0, s, cache_nodes, cache_rows, -1);
  hipLaunchKernelGGL(k_key_place<FREQ>, dim3((unsigned)a.nblk), dim3(CF_THREADS), 0, s, a);
  DG_HIP(hipGetLastError());
  DG_HIP(hipStreamSynchronize(s));
  return DG_OK;
}

extern "C" size_t dg_minhash_workspace_bytes(int64_t m) {
  if (m < 0) return 0;
  KeySort a;
  memset(&a, 0, sizeof(a));
  a.n = m;
  Carve c(nullptr);
  (void)c.take<uint32_t>(64);  // error word
  (void)c.take<int32_t>(64);   // per-sample minima
  carve_keysort(a, c);
  return c.used;
}

extern "C" int dg_minhash_order(const uint64_t *membership, int64_t N, int32_t B,
                                const int32_t *entries, int64_t m, const int32_t *perms,
                                int32_t k, int32_t *order, int32_t *signature, void *ws,
                                size_t ws_bytes, hipStream_t stream) {
  if (!membership || (m > 0 && (!entries || !order)) || (k > 0 && !perms))
    return set_error(DG_EINVAL, "dg_minhash_order: null pointer argument");
  if (N < 1 || N > 0x7fffffffll || B < 1 || B > DG_MAX_BATCHES || m < 0 || k < 1)
    return set_error(DG_EINVAL, "dg_minhash_order: bad sizes");
  const size_t need = dg_minhash_workspace_bytes(m);
  if (!ws || ws_bytes < need || ((uintptr_t)ws & 255))
    return set_error(DG_EWORKSPACE, "dg_minhash_order: workspace needs %zu bytes", need);
  hipStream_t s = stream;
  KeySort a;
  memset(&a, 0, sizeof(a));
  Carve c(ws);
  a.err = c.take<uint32_t>(64);
  int32_t *minv = c.take<int32_t>(64);
  a.mask = membership;
  a.keep = B == 64 ? ~0ull : ((1ull << B) - 1ull);
  a.N = N;
  a.n = m;
  carve_keysort(a, c);
  a.ids = entries;
  a.minv = minv;
  a.order = order;
  a.signature = signature;
  int rc;
  if ((rc = fill_u64(reinterpret_cast<uint64_t *>(a.err), 1, 0, s))) return rc;
  hipLaunchKernelGGL(k_minhash_min, dim3(1), dim3(64), 0, s, perms, k, B, minv, a.err);
  DG_HIP(hipGetLastError());
  int64_t totals[KEYS];
  if ((rc = keysort_count<MINHASH>(a, totals, s))) return rc;
  int64_t run = 0;  // keys ascending; 64 (in no sample) last
  for (int key = 0; key < KEYS; ++key) {
    a.first[key] = run;
    run += totals[key];
  }
  if (a.nblk > 0)
    hipLaunchKernelGGL(k_key_place<MINHASH>, dim3((unsigned)a.nblk), dim3(CF_THREADS), 0, s, a);
  DG_HIP(hipGetLastError());
  uint32_t bits = 0;
  DG_TRY(read_to_host(&bits, a.err, sizeof(bits), s));
  if (bits & ERR_ROW_RANGE)
    return set_error(DG_EINVAL, "dg_minhash_order: a hash value is outside [0, B)");
  if (bits) return set_error(DG_EINVAL, "invalid input data: %s", describe_device_error(bits));
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
