// Feature assembling (DiskGNN §4, Fig. 3, second step): each required feature
// row of a mini-batch comes from the cache table or from the batch's packed
// chunk, at the address the precomputed table gives (§6), written in sampled
// order.  Pure HBM row gather; no lookup structure is consulted.
#include <initializer_list>

#include "dg_rows.h"

namespace dg {
namespace {

constexpr int THREADS = 256;

__device__ __forceinline__ const char *row_source(int32_t l, const char *cache, int64_t cache_rows,
                                                  const char *packed, int64_t packed_rows,
                                                  int64_t row_bytes, int32_t *status) {
  if (l < 0) {
    int64_t r = -(int64_t)l - 1;
    if (r < cache_rows) return cache + r * row_bytes;
  } else if ((int64_t)l < packed_rows) {
    return packed + (int64_t)l * row_bytes;
  }
  if (status) atomicOr(status, 1);
  return nullptr;
}

// The rows of one batch handled by virtual block `blk` of `nblk`.
template <int LPR, int CPL>
__device__ __forceinline__ void assemble16_rows(const v4u *cache, int64_t cache_rows,
                                                const v4u *packed, int64_t packed_rows,
                                                const int32_t *loc, int64_t n, int C, v4u *out,
                                                int32_t *status, int64_t blk, int64_t nblk) {
  constexpr int UNROLL = rows_in_flight(CPL);
  constexpr int GPB = THREADS / LPR;  // row groups per block
  const int sub = threadIdx.x % LPR;
  const int64_t grp = blk * GPB + threadIdx.x / LPR;
  const int64_t ngrp = nblk * GPB;
  for (int64_t j0 = grp * UNROLL; j0 < n; j0 += ngrp * UNROLL) {
    // Every load below is unconditional, at an address that is always valid,
    // and what is not needed is discarded afterwards: with no branch between
    // them, all table entries go out together and then all row vectors.  The
    // table entry of a position past n is read at n - 1.
    int32_t l[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) l[u] = loc[j0 + u < n ? j0 + u : n - 1];
    // scheduling fence (no instruction): no use of an entry is placed between
    // the entry loads, which would make the first one wait alone
    __builtin_amdgcn_sched_barrier(0);
    // Each row's source: the cache table or the packed chunk.  An entry outside
    // both reads the output row it would write (always allocated) instead, is
    // written as zeros, and sets status.
    const v4u *src[UNROLL];
    bool ok[UNROLL];
    bool bad = false;
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int64_t j = j0 + u < n ? j0 + u : n - 1;
      const bool cached = l[u] < 0;
      const int64_t r = cached ? -(int64_t)l[u] - 1 : (int64_t)l[u];
      ok[u] = r < (cached ? cache_rows : packed_rows);
      bad |= j0 + u < n && !ok[u];
      src[u] = ok[u] ? (cached ? cache : packed) + r * C : out + j * C;
    }
    v4u v[UNROLL][CPL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int ch = sub + c * LPR;
        v[u][c] = src[u][ch < C ? ch : C - 1];  // a lane past the row reads its last vector
      }
    if (bad && sub == 0 && status) atomicOr(status, 1);
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
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

template <int LPR, int CPL>
__global__ __launch_bounds__(THREADS) void k_assemble16(const v4u *cache, int64_t cache_rows,
                                                        const v4u *packed, int64_t packed_rows,
                                                        const int32_t *loc, int64_t n, int C,
                                                        v4u *out, int32_t *status) {
  assemble16_rows<LPR, CPL>(cache, cache_rows, packed, packed_rows, loc, n, C, out, status,
                            blockIdx.x, gridDim.x);
}

// Several batches in one launch (each with an output buffer of its own): the
// blocks of batch q are block0[q] .. block0[q+1) - 1, each batch run exactly as
// its own launch would run it.
constexpr int ASM_GROUP = 8;
struct AsmGroup {
  int G;
  int64_t block0[ASM_GROUP + 1];
  const v4u *packed[ASM_GROUP];
  int64_t packed_rows[ASM_GROUP];
  const int32_t *loc[ASM_GROUP];
  int64_t n[ASM_GROUP];
  v4u *out[ASM_GROUP];
};

template <int LPR, int CPL>
__global__ __launch_bounds__(THREADS) void k_assemble16_group(AsmGroup g, const v4u *cache,
                                                              int64_t cache_rows, int C,
                                                              int32_t *status) {
  int q = 0;
#pragma unroll
  for (int k = 1; k < ASM_GROUP; ++k)
    if (k < g.G && (int64_t)blockIdx.x >= g.block0[k]) q = k;
  assemble16_rows<LPR, CPL>(cache, cache_rows, g.packed[q], g.packed_rows[q], g.loc[q], g.n[q],
                            C, g.out[q], status, (int64_t)blockIdx.x - g.block0[q],
                            g.block0[q + 1] - g.block0[q]);
}

// Any row size / alignment: one wave per row, words of sizeof(T).
template <typename T>
__global__ __launch_bounds__(THREADS) void k_assemble_any(const T *cache, int64_t cache_rows,
                                                          const T *packed, int64_t packed_rows,
                                                          const int32_t *loc, int64_t n,
                                                          int64_t W, T *out, int32_t *status) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * THREADS + threadIdx.x) >> 6;
  const int64_t nwave = ((int64_t)gridDim.x * THREADS) >> 6;
  for (int64_t j = wave; j < n; j += nwave) {
    const T *src = reinterpret_cast<const T *>(
        row_source(loc[j], reinterpret_cast<const char *>(cache), cache_rows,
                   reinterpret_cast<const char *>(packed), packed_rows, W * (int64_t)sizeof(T),
                   lane == 0 ? status : nullptr));
    for (int64_t c = lane; c < W; c += 64) out[j * W + c] = src ? src[c] : zero_word<T>();
  }
}

template <typename T>
int launch_any(const void *cache, int64_t cache_rows, const void *packed, int64_t packed_rows,
               const int32_t *loc, int64_t n, int64_t row_bytes, void *out, int32_t *status,
               hipStream_t s) {
  int64_t W = row_bytes / (int64_t)sizeof(T);
  int64_t blocks = (n + 3) / 4;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_assemble_any<T>, dim3((unsigned)blocks), dim3(THREADS), 0, s,
                     (const T *)cache, cache_rows, (const T *)packed, packed_rows, loc, n, W,
                     (T *)out, status);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

template <int LPR, int CPL>
int launch16(const void *cache, int64_t cache_rows, const void *packed, int64_t packed_rows,
             const int32_t *loc, int64_t n, int C, void *out, int32_t *status, hipStream_t s) {
  constexpr int GPB = THREADS / LPR;
  constexpr int UNROLL = rows_in_flight(CPL);
  int64_t groups = (n + UNROLL - 1) / UNROLL;
  int64_t blocks = (groups + GPB - 1) / GPB;
  if (blocks > (1ll << 20)) blocks = 1ll << 20;
  hipLaunchKernelGGL((k_assemble16<LPR, CPL>), dim3((unsigned)blocks), dim3(THREADS), 0, s,
                     (const v4u *)cache, cache_rows, (const v4u *)packed, packed_rows, loc, n, C,
                     (v4u *)out, status);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

bool overlaps(const void *a, int64_t an, const void *b, int64_t bn) {
  if (!a || !b || an <= 0 || bn <= 0) return false;
  uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + (uintptr_t)bn && y < x + (uintptr_t)an;
}

// One batch's arguments, as dg_assemble_batch takes them.
struct AsmArgs {
  const void *packed;
  int64_t packed_rows;
  const int32_t *loc;
  int64_t n;
  void *out;
};

// dg_assemble_batch's argument checks (n == 0 passes: nothing to do).
int check_batch(const void *cache, int64_t cache_rows, const AsmArgs &a, int64_t row_bytes) {
  if (a.n < 0 || row_bytes < 1 || cache_rows < 0 || a.packed_rows < 0)
    return set_error(DG_EINVAL, "dg_assemble_batch: bad sizes");
  if (a.n == 0) return DG_OK;
  if (!a.loc || !a.out || (cache_rows > 0 && !cache) || (a.packed_rows > 0 && !a.packed))
    return set_error(DG_EINVAL, "dg_assemble_batch: null pointer argument");
  const int64_t out_bytes = a.n * row_bytes;
  if (overlaps(a.out, out_bytes, cache, cache_rows * row_bytes) ||
      overlaps(a.out, out_bytes, a.packed, a.packed_rows * row_bytes) ||
      overlaps(a.out, out_bytes, a.loc, a.n * 4))
    return set_error(DG_EINVAL, "dg_assemble_batch: output overlaps an input");
  return DG_OK;
}

// The 16-byte row shape a batch runs with, if it takes that path.
bool shape16(const void *cache, const AsmArgs &a, int64_t row_bytes, RowShape *sh) {
  return word_bytes(row_bytes, {cache, a.packed, a.out}) == 16 && row_shape16(row_bytes / 16, sh);
}

template <int LPR, int CPL>
int64_t blocks16(int64_t n) {
  constexpr int GPB = THREADS / LPR;
  constexpr int UNROLL = rows_in_flight(CPL);
  const int64_t groups = (n + UNROLL - 1) / UNROLL;
  const int64_t blocks = (groups + GPB - 1) / GPB;
  return blocks > (1ll << 20) ? (1ll << 20) : blocks;
}

template <int LPR, int CPL>
int launch16_group(const void *cache, int64_t cache_rows, const AsmArgs *a, int G, int C,
                   int32_t *status, hipStream_t s) {
  AsmGroup g{};
  g.G = G;
  g.block0[0] = 0;
  for (int q = 0; q < G; ++q) {
    g.packed[q] = (const v4u *)a[q].packed;
    g.packed_rows[q] = a[q].packed_rows;
    g.loc[q] = a[q].loc;
    g.n[q] = a[q].n;
    g.out[q] = (v4u *)a[q].out;
    g.block0[q + 1] = g.block0[q] + blocks16<LPR, CPL>(a[q].n);
  }
  hipLaunchKernelGGL((k_assemble16_group<LPR, CPL>), dim3((unsigned)g.block0[G]), dim3(THREADS),
                     0, s, g, (const v4u *)cache, cache_rows, C, status);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

int launch_group(const void *cache, int64_t cache_rows, const AsmArgs *a, int G,
                 int64_t row_bytes, const RowShape &sh, int32_t *status, hipStream_t s) {
  const int C = (int)(row_bytes / 16);
  if (sh.lpr == 4) return launch16_group<4, 1>(cache, cache_rows, a, G, C, status, s);
  if (sh.lpr == 8) return launch16_group<8, 1>(cache, cache_rows, a, G, C, status, s);
  if (sh.lpr == 16) return launch16_group<16, 1>(cache, cache_rows, a, G, C, status, s);
  if (sh.lpr == 32 && sh.cpl == 1) return launch16_group<32, 1>(cache, cache_rows, a, G, C, status, s);
  if (sh.lpr == 64 && sh.cpl == 1) return launch16_group<64, 1>(cache, cache_rows, a, G, C, status, s);
  if (sh.lpr == 64 && sh.cpl == 2) return launch16_group<64, 2>(cache, cache_rows, a, G, C, status, s);
  return launch16_group<64, 4>(cache, cache_rows, a, G, C, status, s);
}

}  // namespace
}  // namespace dg

using namespace dg;

extern "C" int dg_assemble_batch(const void *cache, int64_t cache_rows, const void *packed_b,
                                 int64_t packed_rows_b, const int32_t *loc_b, int64_t n_b,
                                 int64_t row_bytes, void *out, int32_t *status,
                                 hipStream_t stream) {
  if (n_b < 0 || row_bytes < 1 || cache_rows < 0 || packed_rows_b < 0)
    return set_error(DG_EINVAL, "dg_assemble_batch: bad sizes");
  if (n_b == 0) return DG_OK;
  if (!loc_b || !out || (cache_rows > 0 && !cache) || (packed_rows_b > 0 && !packed_b))
    return set_error(DG_EINVAL, "dg_assemble_batch: null pointer argument");
  const int64_t out_bytes = n_b * row_bytes;
  if (overlaps(out, out_bytes, cache, cache_rows * row_bytes) ||
      overlaps(out, out_bytes, packed_b, packed_rows_b * row_bytes) ||
      overlaps(out, out_bytes, loc_b, n_b * 4))
    return set_error(DG_EINVAL, "dg_assemble_batch: output overlaps an input");
  const int w = word_bytes(row_bytes, {cache, packed_b, out});
  if (w == 16) {
    const int64_t C = row_bytes / 16;
    RowShape sh;
    if (row_shape16(C, &sh)) {
      const int c = (int)C;
      if (sh.lpr == 4) return launch16<4, 1>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, c, out, status, stream);
      if (sh.lpr == 8) return launch16<8, 1>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, c, out, status, stream);
      if (sh.lpr == 16) return launch16<16, 1>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, c, out, status, stream);
      if (sh.lpr == 32 && sh.cpl == 1) return launch16<32, 1>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, c, out, status, stream);
      if (sh.lpr == 64 && sh.cpl == 1) return launch16<64, 1>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, c, out, status, stream);
      if (sh.lpr == 64 && sh.cpl == 2) return launch16<64, 2>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, c, out, status, stream);
      if (sh.lpr == 64 && sh.cpl == 4) return launch16<64, 4>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, c, out, status, stream);
    }
    return launch_any<uint4>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, row_bytes, out, status, stream);
  }
  if (w == 8) return launch_any<uint2>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, row_bytes, out, status, stream);
  if (w == 4) return launch_any<uint32_t>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, row_bytes, out, status, stream);
  if (w == 2) return launch_any<uint16_t>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, row_bytes, out, status, stream);
  return launch_any<uint8_t>(cache, cache_rows, packed_b, packed_rows_b, loc_b, n_b, row_bytes, out, status, stream);
}

extern "C" int dg_assemble_batches(const void *cache, int64_t cache_rows, const void *packed,
                                   const int64_t *packed_ptr_host, const int32_t *loc,
                                   int64_t loc_stride, const int64_t *node_count, int32_t B,
                                   int64_t row_bytes, void *const *outs, int32_t n_outs,
                                   int32_t *status, hipStream_t stream) {
  if (B < 0 || n_outs < 1 || !outs || (B > 0 && (!packed_ptr_host || !node_count)) ||
      row_bytes < 1 || loc_stride < 0)
    return set_error(DG_EINVAL, "dg_assemble_batches: bad argument");
  for (int32_t b = 0; b < B; ++b) {  // every batch is checked before any launch
    const int64_t p0 = packed_ptr_host[b], p1 = packed_ptr_host[b + 1];
    const int64_t n = node_count[b];
    if (p0 < 0 || p1 < p0 || n < 0 || n > loc_stride)
      return set_error(DG_EINVAL, "dg_assemble_batches: batch %d: bad chunk bounds or n_b", b);
  }
  // Consecutive batches with output buffers of their own (outs[b % n_outs]
  // distinct and apart) share one launch, up to ASM_GROUP of them, when they
  // take the 16-byte path: each batch is still checked as dg_assemble_batch
  // checks it, in batch order, before its launch.
  auto args_of = [&](int32_t b) {
    const int64_t p0 = packed_ptr_host[b], p1 = packed_ptr_host[b + 1];
    AsmArgs a;
    a.packed = (p1 > p0 && packed) ? static_cast<const char *>(packed) + p0 * row_bytes : nullptr;
    a.packed_rows = p1 - p0;
    a.loc = loc ? loc + (int64_t)b * loc_stride : nullptr;
    a.n = node_count[b];
    a.out = outs[b % n_outs];
    return a;
  };
  for (int32_t b = 0; b < B;) {
    AsmArgs a[ASM_GROUP];
    a[0] = args_of(b);
    int rc = check_batch(cache, cache_rows, a[0], row_bytes);
    if (rc != DG_OK) return rc;
    RowShape sh{};
    int G = 1;
    if (a[0].n > 0 && shape16(cache, a[0], row_bytes, &sh)) {
      while (G < ASM_GROUP && G < n_outs && b + G < B) {
        const AsmArgs c = args_of(b + G);
        RowShape sc{};
        bool apart = c.n > 0 && shape16(cache, c, row_bytes, &sc) && sc.lpr == sh.lpr &&
                     sc.cpl == sh.cpl;
        for (int q = 0; apart && q < G; ++q)
          apart = !overlaps(c.out, c.n * row_bytes, a[q].out, a[q].n * row_bytes) &&
                  !overlaps(c.out, c.n * row_bytes, a[q].loc, a[q].n * 4) &&
                  !overlaps(c.out, c.n * row_bytes, a[q].packed, a[q].packed_rows * row_bytes) &&
                  !overlaps(a[q].out, a[q].n * row_bytes, c.loc, c.n * 4) &&
                  !overlaps(a[q].out, a[q].n * row_bytes, c.packed, c.packed_rows * row_bytes);
        if (!apart || check_batch(cache, cache_rows, c, row_bytes) != DG_OK) break;
        a[G++] = c;
      }
    }
    if (G > 1) {
      if ((rc = launch_group(cache, cache_rows, a, G, row_bytes, sh, status, stream)))
        return rc;
    } else {
      rc = dg_assemble_batch(cache, cache_rows, a[0].packed, a[0].packed_rows, a[0].loc, a[0].n,
                             row_bytes, a[0].out, status, stream);
      if (rc != DG_OK) return rc;
    }
    b += G;
  }
  return DG_OK;
}
