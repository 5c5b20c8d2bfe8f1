// The fan-out gather of batched packing (DiskGNN §5.2, Fig. 6b): each row of
// the group's non-cached unique set is read once from the feature table and
// written to every packed row that holds it, and (with a cache table) the
// cache rows are filled in the same launch, the cache taken as one more
// mini-batch.
#include <initializer_list>

#include "dg_rows.h"

namespace dg {
namespace {

constexpr int THREADS = 256;

// Fan-out gather, 16-byte path: a group of LPR lanes reads the row of one U_nc
// node once and stores it into each of its destination rows.  Every U_nc node
// has at least one destination; its first destination index is loaded together
// with the row, so the common single-destination case needs two dependent
// round trips (indices, then row + destination) before its stores.
// Items n_unc .. n_unc + n_cache - 1 fill the cache table, the cache taken as
// one more mini-batch of the same pass: item n_unc + s copies the row of
// cache_nodes[s] into cache row s (a slot holding -1 is left as it is; an ID
// outside [0, N) is reported and its row left as it is).
template <int LPR, int CPL>
__global__ __launch_bounds__(THREADS) void k_fanout16(const v4u *X, int64_t N,
                                                      const int32_t *unc_ids,
                                                      const int64_t *unc_off, int64_t n_unc,
                                                      int64_t n_pairs, const int64_t *pairdest,
                                                      int C, v4u *packed,
                                                      const int32_t *cache_nodes,
                                                      int64_t n_cache, v4u *cache_table,
                                                      uint32_t *err) {
  constexpr int UNROLL = rows_in_flight(CPL);
  constexpr int GPB = THREADS / LPR;
  const int sub = threadIdx.x % LPR;
  const int64_t grp = (int64_t)blockIdx.x * GPB + threadIdx.x / LPR;
  const int64_t ngrp = (int64_t)gridDim.x * GPB;
  const int64_t n_items = n_unc + n_cache;
  for (int64_t i0 = grp * UNROLL; i0 < n_items; i0 += ngrp * UNROLL) {
    int64_t p0[UNROLL], p1[UNROLL], d0[UNROLL];
    int32_t id[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int64_t i = i0 + u;
      p0[u] = p1[u] = 0;
      id[u] = -1;
      if (i < n_unc) {
        id[u] = unc_ids[i];
        p0[u] = unc_off[i];
        p1[u] = i + 1 < n_unc ? unc_off[i + 1] : n_pairs;
      } else if (i < n_items) {
        const int32_t v = cache_nodes[i - n_unc];
        if (v >= 0 && (int64_t)v < N) id[u] = v;
        else if (v != -1 && sub == 0) atomicOr(err, ERR_NODE_RANGE);
      }
    }
    v4u v[UNROLL][CPL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      d0[u] = p1[u] > p0[u] ? pairdest[p0[u]] : -1;
      const v4u *src = id[u] >= 0 ? X + (int64_t)id[u] * C : nullptr;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int ch = sub + c * LPR;
        v[u][c] = (src && ch < C) ? ld_stream(src + ch) : v4u{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int64_t i = i0 + u;
      v4u *dst;
      if (i >= n_unc) {  // a cache row
        if (i >= n_items || id[u] < 0) continue;
        dst = cache_table + (i - n_unc) * C;
      } else {
        if (d0[u] < 0) continue;
        dst = packed + d0[u] * C;
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int ch = sub + c * LPR;
        if (ch < C) st_stream(v[u][c], dst + ch);
      }
      for (int64_t p = p0[u] + 1; p < p1[u]; ++p) {
        dst = packed + pairdest[p] * C;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const int ch = sub + c * LPR;
          if (ch < C) st_stream(v[u][c], dst + ch);
        }
      }
    }
  }
}

// Any row size / alignment: one wave per item (U_nc node, then cache row), words
// of sizeof(T).
template <typename T>
__global__ __launch_bounds__(THREADS) void k_fanout_any(const T *X, int64_t N,
                                                        const int32_t *unc_ids,
                                                        const int64_t *unc_off, int64_t n_unc,
                                                        int64_t n_pairs, const int64_t *pairdest,
                                                        int64_t W, T *packed,
                                                        const int32_t *cache_nodes,
                                                        int64_t n_cache, T *cache_table,
                                                        uint32_t *err) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * THREADS + threadIdx.x) >> 6;
  const int64_t nwave = ((int64_t)gridDim.x * THREADS) >> 6;
  for (int64_t i = wave; i < n_unc + n_cache; i += nwave) {
    if (i >= n_unc) {
      const int64_t s = i - n_unc;
      const int32_t v = cache_nodes[s];
      if (v < 0 || (int64_t)v >= N) {
        if (v != -1 && lane == 0) atomicOr(err, ERR_NODE_RANGE);
        continue;
      }
      for (int64_t c = lane; c < W; c += 64) cache_table[s * W + c] = X[(int64_t)v * W + c];
      continue;
    }
    const T *src = X + (int64_t)unc_ids[i] * W;
    int64_t p0 = unc_off[i], p1 = i + 1 < n_unc ? unc_off[i + 1] : n_pairs;
    for (int64_t c = lane; c < W; c += 64) {
      T x = src[c];
      for (int64_t p = p0; p < p1; ++p) packed[pairdest[p] * W + c] = x;
    }
  }
}


template <int LPR, int CPL>
void launch16(const RowCopy &r, int C, hipStream_t s) {
  constexpr int GPB = THREADS / LPR;
  constexpr int UNROLL = rows_in_flight(CPL);
  int64_t groups = (r.n + r.n_cache + UNROLL - 1) / UNROLL;
  int64_t blocks = (groups + GPB - 1) / GPB;
  if (blocks > (1ll << 20)) blocks = 1ll << 20;
  hipLaunchKernelGGL((k_fanout16<LPR, CPL>), dim3((unsigned)blocks), dim3(THREADS), 0, s,
                     (const v4u *)r.X, r.N, r.ids, r.off, r.n, r.pairs, r.dest, C,
                     (v4u *)r.packed, r.cache_nodes, r.n_cache, (v4u *)r.cache_table, r.err);
}

template <typename T>
void launch_any(const RowCopy &r, hipStream_t s) {
  int64_t blocks = (r.n + r.n_cache + 3) / 4;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_fanout_any<T>, dim3((unsigned)blocks), dim3(THREADS), 0, s,
                     (const T *)r.X, r.N, r.ids, r.off, r.n, r.pairs, r.dest,
                     r.row_bytes / (int64_t)sizeof(T), (T *)r.packed, r.cache_nodes, r.n_cache,
                     (T *)r.cache_table, r.err);
}

}  // namespace

int launch_fanout(const RowCopy &r, hipStream_t s) {
  if (r.n + r.n_cache == 0) return DG_OK;
  const int w = word_bytes(r.row_bytes, {r.X, r.packed, r.cache_table});
  RowShape sh;
  if (w == 16 && row_shape16(r.row_bytes / 16, &sh)) {
    const int C = (int)(r.row_bytes / 16);
    if (sh.lpr == 4) launch16<4, 1>(r, C, s);
    else if (sh.lpr == 8) launch16<8, 1>(r, C, s);
    else if (sh.lpr == 16) launch16<16, 1>(r, C, s);
    else if (sh.lpr == 32 && sh.cpl == 1) launch16<32, 1>(r, C, s);
    else if (sh.lpr == 64 && sh.cpl == 1) launch16<64, 1>(r, C, s);
    else if (sh.lpr == 64 && sh.cpl == 2) launch16<64, 2>(r, C, s);
    else launch16<64, 4>(r, C, s);
  } else if (w == 16) {
    launch_any<uint4>(r, s);
  } else if (w == 8) {
    launch_any<uint2>(r, s);
  } else if (w == 4) {
    launch_any<uint32_t>(r, s);
  } else if (w == 2) {
    launch_any<uint16_t>(r, s);
  } else {
    launch_any<uint8_t>(r, s);
  }
  DG_HIP(hipGetLastError());
  return DG_OK;
}

}  // namespace dg
