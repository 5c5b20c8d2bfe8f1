// Shared machinery of libdg: error reporting, fills, prefix scans and the
// node-major membership-mask compaction used by sampling (per-hop new-node
// lists) and packing (group unique set, per-batch packed order).
#include <stdarg.h>
#include <string.h>

#include "dg_common.h"

namespace dg {

static thread_local char g_err[512] = "";

int set_error(int status, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return status;
}

const char *describe_device_error(uint32_t bits) {
  if (bits & ERR_NODE_RANGE) return "a node ID is outside [0, N)";
  if (bits & ERR_DUP_NODE) return "a node appears twice in one mini-batch";
  if (bits & ERR_CSR) return "CSR offsets are decreasing or outside [0, num_edges]";
  if (bits & ERR_NBR_RANGE) return "a CSR neighbour ID is outside [0, N)";
  if (bits & ERR_CACHE_SLOT) return "cache_slot holds a value below -1";
  if (bits & ERR_ROW_RANGE) return "an address-table entry is outside its table";
  return "unknown device error";
}

// ---------------------------------------------------------------- fill
__global__ void k_fill_u64(uint64_t *p, size_t n, uint64_t v) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = v;
}

int fill_u64(uint64_t *p, size_t n, uint64_t value, hipStream_t s) {
  if (n == 0) return DG_OK;
  size_t blocks = (n + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_fill_u64, dim3((unsigned)blocks), dim3(256), 0, s, p, n, value);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

// ---------------------------------------------------------------- scan
constexpr int SC_THREADS = 256;
constexpr int SC_ITEMS = 8;
constexpr int SC_TILE = SC_THREADS * SC_ITEMS;

size_t scan_tile_count(int64_t n) { return (size_t)((n + SC_TILE - 1) / SC_TILE) + 1; }

// Block-wide exclusive scan of one value per thread; *total gets the block sum.
template <int NT>
__device__ __forceinline__ int64_t block_excl_scan(int64_t x, int64_t *total) {
  __shared__ int64_t s_w[NT / 64];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  int64_t incl = wave_incl_sum(x);
  if (lane == 63) s_w[w] = incl;
  __syncthreads();
  int64_t before = 0, sum = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) {
    int64_t v = s_w[i];
    if (i < w) before += v;
    sum += v;
  }
  __syncthreads();
  *total = sum;
  return before + incl - x;
}

__global__ __launch_bounds__(SC_THREADS) void k_scan_reduce(const int64_t *in, int64_t n,
                                                            int64_t *tile_sums) {
  int64_t t0 = (int64_t)blockIdx.x * SC_TILE;
  int64_t acc = 0;
#pragma unroll
  for (int r = 0; r < SC_ITEMS; ++r) {
    int64_t i = t0 + r * SC_THREADS + threadIdx.x;
    if (i < n) acc += in[i];
  }
  int64_t total;
  (void)block_excl_scan<SC_THREADS>(acc, &total);
  if (threadIdx.x == 0) tile_sums[blockIdx.x] = total;
}

// One block scans the tile sums in place (exclusive); tile_sums[ntiles] = total.
__global__ __launch_bounds__(1024) void k_scan_tiles(int64_t *tile_sums, int64_t ntiles) {
  int64_t carry = 0;
  for (int64_t c0 = 0; c0 < ntiles; c0 += 1024) {
    int64_t i = c0 + threadIdx.x;
    int64_t v = i < ntiles ? tile_sums[i] : 0;
    int64_t total;
    int64_t ex = block_excl_scan<1024>(v, &total);
    if (i < ntiles) tile_sums[i] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) tile_sums[ntiles] = carry;
}

// Each thread owns SC_ITEMS consecutive items of the tile.
__global__ __launch_bounds__(SC_THREADS) void k_scan_apply(const int64_t *in, int64_t *out,
                                                           int64_t n, const int64_t *tile_sums) {
  int64_t t0 = (int64_t)blockIdx.x * SC_TILE + (int64_t)threadIdx.x * SC_ITEMS;
  int64_t v[SC_ITEMS];
  int64_t acc = 0;
#pragma unroll
  for (int r = 0; r < SC_ITEMS; ++r) {
    int64_t i = t0 + r;
    v[r] = i < n ? in[i] : 0;
    acc += v[r];
  }
  int64_t total;
  int64_t run = tile_sums[blockIdx.x] + block_excl_scan<SC_THREADS>(acc, &total);
#pragma unroll
  for (int r = 0; r < SC_ITEMS; ++r) {
    int64_t i = t0 + r;
    if (i < n) out[i] = run;
    run += v[r];
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) {
    int64_t ntiles = gridDim.x;
    out[n] = tile_sums[ntiles];
  }
}

int scan_exclusive(const int64_t *in, int64_t *out, int64_t n, int64_t *tile_sums,
                   hipStream_t s) {
  int64_t ntiles = (n + SC_TILE - 1) / SC_TILE;
  if (ntiles == 0) {
    DG_HIP(hipMemsetAsync(out, 0, sizeof(int64_t), s));
    return DG_OK;
  }
  hipLaunchKernelGGL(k_scan_reduce, dim3((unsigned)ntiles), dim3(SC_THREADS), 0, s, in, n,
                     tile_sums);
  hipLaunchKernelGGL(k_scan_tiles, dim3(1), dim3(1024), 0, s, tile_sums, ntiles);
  hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)ntiles), dim3(SC_THREADS), 0, s, in, out, n,
                     tile_sums);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

// ---------------------------------------------------------------- mask compaction
size_t mask_scan_ws_bytes(int64_t N, int B) {
  Carve c(nullptr);
  MaskScan m{};
  m.N = N;
  m.B = B;
  mask_scan_carve(m, c);
  return c.used;
}

void mask_scan_carve(MaskScan &m, Carve &c) {
  m.nblk = mc_blocks(m.N);
  size_t cells = (size_t)mc_rows(m.B) * (size_t)m.nblk;
  m.cnt = c.take<uint32_t>(cells);
  m.base = c.take<int64_t>(cells);
  m.totals = c.take<int64_t>((size_t)mc_rows(m.B));
}

// Count pass: for each tile, the number of members of every batch (non-cached
// only), of U, of U_nc, and of U_nc's (node, batch) pairs.
__global__ __launch_bounds__(MC_THREADS) void k_mask_count(MaskScan a) {
  __shared__ uint32_t s_cnt[DG_MAX_BATCHES + 3];
  const int B = a.B, rows = mc_rows(B);
  for (int i = threadIdx.x; i < rows; i += MC_THREADS) s_cnt[i] = 0;
  __syncthreads();
  const int lane = lane_id();
  const int64_t t0 = (int64_t)blockIdx.x * MC_TILE;
  for (int r = 0; r < MC_ROUNDS; ++r) {
    int64_t u = t0 + (int64_t)r * MC_THREADS + threadIdx.x;
    uint64_t m = u < a.N ? a.mask[u] : 0ull;
    uint64_t any = __ballot(m != 0ull);
    if (any == 0ull) continue;  // wave-uniform
    bool cached = false;
    if (m != 0ull && a.cache_slot) {
      int32_t sl = a.cache_slot[u];
      if (sl < -1) atomicOr(a.err, ERR_CACHE_SLOT);
      cached = sl >= 0;
    }
    uint64_t mnc = cached ? 0ull : m;
    uint64_t anync = __ballot(mnc != 0ull);
    if (lane == 0) {
      atomicAdd(&s_cnt[row_all(B)], (uint32_t)__popcll(any));
      atomicAdd(&s_cnt[row_packed(B)], (uint32_t)__popcll(anync));
    }
    uint64_t uni = wave_or(mnc);
    while (uni) {
      int b = __ffsll((long long)uni) - 1;
      uni &= uni - 1;
      uint64_t bal = __ballot((mnc >> b) & 1ull);
      if (lane == 0) atomicAdd(&s_cnt[b], (uint32_t)__popcll(bal));
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t pairs = 0;
    for (int b = 0; b < B; ++b) pairs += s_cnt[b];
    s_cnt[row_pairs(B)] = pairs;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < rows; i += MC_THREADS)
    a.cnt[(size_t)i * a.nblk + blockIdx.x] = s_cnt[i];
}

// One block per row: exclusive scan of the row's per-tile counts.
__global__ __launch_bounds__(1024) void k_mask_rows(MaskScan a) {
  const int row = blockIdx.x;
  const uint32_t *c = a.cnt + (size_t)row * a.nblk;
  int64_t *o = a.base + (size_t)row * a.nblk;
  int64_t carry = 0;
  for (int64_t c0 = 0; c0 < a.nblk; c0 += 1024) {
    int64_t i = c0 + threadIdx.x;
    int64_t v = i < a.nblk ? (int64_t)c[i] : 0;
    int64_t total;
    int64_t ex = block_excl_scan<1024>(v, &total);
    if (i < a.nblk) o[i] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) a.totals[row] = carry;
}

int mask_scan_count(MaskScan &m, int64_t *host_totals, hipStream_t s) {
  if (m.nblk == 0) {
    for (int i = 0; i < mc_rows(m.B); ++i) host_totals[i] = 0;
    return DG_OK;
  }
  hipLaunchKernelGGL(k_mask_count, dim3((unsigned)m.nblk), dim3(MC_THREADS), 0, s, m);
  hipLaunchKernelGGL(k_mask_rows, dim3((unsigned)mc_rows(m.B)), dim3(1024), 0, s, m);
  DG_HIP(hipGetLastError());
  DG_HIP(hipMemcpyAsync(host_totals, m.totals, sizeof(int64_t) * mc_rows(m.B),
                        hipMemcpyDeviceToHost, s));
  DG_HIP(hipStreamSynchronize(s));
  return DG_OK;
}

// Write pass.  Within a tile, round r covers nodes t0 + r*256 + [0,256), so
// ascending (round, wave, lane) order is ascending node order; ranks come from
// per-wave ballots plus the counts of earlier waves and rounds.
__global__ __launch_bounds__(MC_THREADS) void k_mask_write(MaskScan a) {
  __shared__ int64_t s_run[DG_MAX_BATCHES + 3];
  __shared__ int64_t s_w[MC_THREADS / 64][DG_MAX_BATCHES + 3];
  const int B = a.B, rows = mc_rows(B);
  const int lane = lane_id(), w = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < rows; i += MC_THREADS)
    s_run[i] = a.base[(size_t)i * a.nblk + blockIdx.x];
  const int64_t t0 = (int64_t)blockIdx.x * MC_TILE;
  for (int r = 0; r < MC_ROUNDS; ++r) {
    for (int i = threadIdx.x; i < (MC_THREADS / 64) * rows; i += MC_THREADS)
      s_w[i / rows][i % rows] = 0;
    __syncthreads();
    int64_t u = t0 + (int64_t)r * MC_THREADS + threadIdx.x;
    uint64_t m = u < a.N ? a.mask[u] : 0ull;
    uint64_t any = __ballot(m != 0ull);
    uint64_t mnc = 0ull, anync = 0ull, uni = 0ull;
    int64_t pc = 0, pincl = 0;
    if (any != 0ull) {
      bool cached = (m != 0ull && a.cache_slot) ? a.cache_slot[u] >= 0 : false;
      mnc = cached ? 0ull : m;
      anync = __ballot(mnc != 0ull);
      pc = __popcll(mnc);
      pincl = wave_incl_sum(pc);
      uni = wave_or(mnc);
      if (lane == 0) {
        s_w[w][row_all(B)] = __popcll(any);
        s_w[w][row_packed(B)] = __popcll(anync);
      }
      if (lane == 63) s_w[w][row_pairs(B)] = pincl;
      uint64_t x = uni;
      while (x) {
        int b = __ffsll((long long)x) - 1;
        x &= x - 1;
        uint64_t bal = __ballot((mnc >> b) & 1ull);
        if (lane == 0) s_w[w][b] = __popcll(bal);
      }
    }
    __syncthreads();
    if (any != 0ull) {
      const uint64_t lt = lanes_below();
      auto wave_base = [&](int row) {
        int64_t v = s_run[row];
        for (int i = 0; i < w; ++i) v += s_w[i][row];
        return v;
      };
      if (m != 0ull && a.uniq_out)
        a.uniq_out[wave_base(row_all(B)) + __popcll(any & lt)] = (int32_t)u;
      int64_t pair0 = wave_base(row_pairs(B)) + (pincl - pc);
      if (mnc != 0ull) {
        int64_t rk = wave_base(row_packed(B)) + __popcll(anync & lt);
        if (a.unc_ids) a.unc_ids[rk] = (int32_t)u;
        if (a.unc_off) a.unc_off[rk] = pair0;
        if (a.nodeoff) a.nodeoff[u] = pair0;
      }
      uint64_t x = uni;
      while (x) {
        int b = __ffsll((long long)x) - 1;
        x &= x - 1;
        uint64_t bal = __ballot((mnc >> b) & 1ull);
        if ((mnc >> b) & 1ull) {
          int64_t dest = a.seg_base[b] + wave_base(b) + __popcll(bal & lt);
          if (a.seg_out) a.seg_out[dest] = (int32_t)u;
          if (a.pairdest) a.pairdest[pair0 + __popcll(mnc & ((1ull << b) - 1ull))] = dest;
        }
      }
      if (a.clear && m != 0ull) a.mask[u] = 0ull;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < rows; i += MC_THREADS) {
      int64_t add = 0;
      for (int j = 0; j < MC_THREADS / 64; ++j) add += s_w[j][i];
      s_run[i] += add;
    }
    __syncthreads();
  }
}

int mask_scan_write(const MaskScan &m, hipStream_t s) {
  if (m.nblk == 0) return DG_OK;
  hipLaunchKernelGGL(k_mask_write, dim3((unsigned)m.nblk), dim3(MC_THREADS), 0, s, m);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

}  // namespace dg

extern "C" const char *dg_last_error(void) { return dg::g_err; }
extern "C" const char *dg_version(void) { return "libdg 0.1 (gfx950)"; }
