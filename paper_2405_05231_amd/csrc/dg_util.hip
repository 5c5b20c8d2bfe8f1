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
  if (bits & ERR_INTERNAL) return "internal table overflow";
  if (bits & ERR_MEMBERSHIP) return "the membership mask does not match the node lists";
  return "unknown device error";
}

// ---------------------------------------------------------------- host reads
constexpr size_t STAGE_BYTES = 4096;

int read_to_host(void *dst, const void *src, size_t bytes, hipStream_t s) {
  static thread_local void *stage = nullptr;
  static thread_local bool tried = false;
  if (!tried) {
    tried = true;
    if (hipHostMalloc(&stage, STAGE_BYTES, hipHostMallocDefault) != hipSuccess) {
      (void)hipGetLastError();
      stage = nullptr;
    }
  }
  if (stage && bytes <= STAGE_BYTES) {
    DG_HIP(hipMemcpyAsync(stage, src, bytes, hipMemcpyDeviceToHost, s));
    DG_HIP(hipStreamSynchronize(s));
    memcpy(dst, stage, bytes);
    return DG_OK;
  }
  DG_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s));
  DG_HIP(hipStreamSynchronize(s));
  return DG_OK;
}

// ---------------------------------------------------------------- side stream
int side_stream(SideStream **out) {
  constexpr int MAX_DEV = 16;
  static thread_local SideStream ss[MAX_DEV];
  static thread_local bool made[MAX_DEV] = {};
  int dev = 0;
  DG_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= MAX_DEV) return set_error(DG_EHIP, "device index %d out of range", dev);
  if (!made[dev]) {
    DG_HIP(hipStreamCreateWithFlags(&ss[dev].s, hipStreamNonBlocking));
    DG_HIP(hipEventCreateWithFlags(&ss[dev].fork, hipEventDisableTiming));
    DG_HIP(hipEventCreateWithFlags(&ss[dev].join, hipEventDisableTiming));
    made[dev] = true;
  }
  *out = &ss[dev];
  return DG_OK;
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
  size_t rows = (size_t)mc_rows(m.B);
  m.cnt = c.take<uint32_t>(rows * (size_t)m.nblk);
  m.wpre = c.take<uint32_t>(rows * (size_t)m.nblk * MC_WAVES);
  m.wcnt = c.take<uint32_t>((size_t)m.nblk * MC_WAVES);
  m.cw_mask = c.take<uint64_t>((size_t)m.nblk * MC_BLOCK_NODES);
  m.cw_off = c.take<uint16_t>((size_t)m.nblk * MC_BLOCK_NODES);
  m.base = c.take<int64_t>(rows * (size_t)m.nblk);
  m.chunk_sum = c.take<int64_t>(rows * (size_t)mc_chunks(m.nblk));
  m.totals = c.take<int64_t>(rows + 1);  // + a slot for the staged error word
}

// Tile loads: all MC_ROUNDS mask words (and the prev words and cached flags of
// non-empty ones) are requested before any is used, so a wave keeps 16 loads in
// flight.
struct TileBits {
  uint64_t m[MC_ROUNDS];
  uint32_t cached;  // bit r: node of round r is cached
};

// With update_prev, prev takes the listed bits as soon as they are known
// (prev |= the new bits; the word is owned by this lane), so no second load is
// needed later.
__device__ __forceinline__ void load_tile(const MaskScan &a, int64_t t0, int lane, TileBits &t,
                                          bool check_slots, bool update_prev) {
  uint32_t live = 0xffffu;  // bit r: round r may hold bits to list
  if (a.touched) {
    const uint8_t *f = a.touched + (t0 >> 6);
    live = 0;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) live |= (f[r] ? 1u : 0u) << r;
  }
#pragma unroll
  for (int r = 0; r < MC_ROUNDS; ++r) {
    int64_t u = t0 + r * 64 + lane;
    t.m[r] = (u < a.N && ((live >> r) & 1u)) ? a.mask[u] : 0ull;
  }
  if (a.B < 64) {  // bits of batches outside the group are ignored
    const uint64_t keep = (1ull << a.B) - 1ull;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) t.m[r] &= keep;
  }
  if (a.prev) {
    uint64_t p[MC_ROUNDS];
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) p[r] = t.m[r] ? a.prev[t0 + r * 64 + lane] : 0ull;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) {
      t.m[r] &= ~p[r];
      if (update_prev && t.m[r] != 0ull) a.prev[t0 + r * 64 + lane] = p[r] | t.m[r];
    }
  }
  t.cached = 0;
  if (a.cache_slot) {
    int32_t sl[MC_ROUNDS];
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r)
      sl[r] = t.m[r] ? a.cache_slot[t0 + r * 64 + lane] : -1;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) {
      if (check_slots && sl[r] < -1) atomicOr(a.err, ERR_CACHE_SLOT);
      t.cached |= (sl[r] >= 0 ? 1u : 0u) << r;
    }
  }
}

// Per-wave counts of one tile: lane b returns batch b's non-cached members;
// *cu, *cnc, *cp, *call (wave-uniform) get the members of U, of U_nc, U_nc's
// pairs and all pairs.  Per-batch counts walk the tile's non-empty words one at
// a time: the word is read out of its lane (v_readlane), and lane b tests bit b,
// so the work follows the words present rather than the batches they touch.
__device__ __forceinline__ uint32_t tile_counts(const TileBits &t, int lane, uint32_t *cu,
                                                uint32_t *cnc, uint32_t *cp, uint32_t *call) {
  uint32_t mine = 0, u = 0, nc = 0;
  int32_t pl = 0, al = 0;  // this lane's pair counts (U_nc pairs, all pairs)
#pragma unroll
  for (int r = 0; r < MC_ROUNDS; ++r) {
    const uint64_t m = t.m[r];
    const uint64_t any = __ballot(m != 0ull);
    if (any == 0ull) continue;  // wave-uniform
    const uint64_t mnc = ((t.cached >> r) & 1u) ? 0ull : m;
    al += __popcll(m);
    pl += __popcll(mnc);
    u += (uint32_t)__popcll(any);
    uint64_t anc = __ballot(mnc != 0ull);
    nc += (uint32_t)__popcll(anc);
    while (anc) {
      const int l = __ffsll((long long)anc) - 1;
      anc &= anc - 1;
      const uint64_t w = (uint64_t)read_lane((int64_t)mnc, l);
      mine += (uint32_t)((w >> lane) & 1ull);
    }
  }
  *cu = u;
  *cnc = nc;
  *cp = (uint32_t)__ockl_wfred_add_i32(pl);
  *call = (uint32_t)__ockl_wfred_add_i32(al);
  return mine;
}

// Count pass: per block, the number of members of every batch (non-cached
// only), of U, of U_nc, and of U_nc's (node, batch) pairs; stored as one
// contiguous row per block, plus each wave's exclusive prefix within the block
// (so the write pass does not count again).
__global__ __launch_bounds__(MC_THREADS) void k_mask_count(MaskScan a) {
  __shared__ uint32_t s_cnt[MC_WAVES][DG_MAX_BATCHES + 4];
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const int B = a.B, rows = mc_rows(B);
  const int64_t t0 = (int64_t)blockIdx.x * MC_BLOCK_NODES + (int64_t)w * MC_TILE;
  TileBits t;
  load_tile(a, t0, lane, t, true, a.keep_prev);
  uint32_t cu, cnc, cp, call;
  uint32_t mine = tile_counts(t, lane, &cu, &cnc, &cp, &call);
  // the tile's non-empty words, in node order, for the write pass
  {
    const size_t gw = ((size_t)blockIdx.x * MC_WAVES + w) * MC_TILE;
    const uint64_t lt = lanes_below();
    uint32_t run = 0;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) {
      const uint64_t any = __ballot(t.m[r] != 0ull);
      if (any == 0ull) continue;
      if (t.m[r] != 0ull) {
        const size_t at = gw + run + (uint32_t)__popcll(any & lt);
        a.cw_mask[at] = t.m[r];
        a.cw_off[at] = (uint16_t)((r * 64 + lane) | ((int)((t.cached >> r) & 1u) << 15));
      }
      run += (uint32_t)__popcll(any);
    }
    if (lane == 0) a.wcnt[(size_t)blockIdx.x * MC_WAVES + w] = run;
  }
  if (lane < B) s_cnt[w][lane] = mine;
  if (lane == 0) {
    s_cnt[w][row_all(B)] = cu;
    s_cnt[w][row_packed(B)] = cnc;
    s_cnt[w][row_pairs(B)] = cp;
    s_cnt[w][row_all_pairs(B)] = call;
  }
  __syncthreads();
  uint32_t *pre = a.wpre + (size_t)blockIdx.x * MC_WAVES * rows;
  for (int i = threadIdx.x; i < rows; i += MC_THREADS) {
    uint32_t v = 0;
#pragma unroll
    for (int j = 0; j < MC_WAVES; ++j) {
      pre[j * rows + i] = v;
      v += s_cnt[j][i];
    }
    a.cnt[(size_t)blockIdx.x * rows + i] = v;
  }
}

// Row scan, three phases over the [nblk][rows] count matrix: chunk sums,
// scan of chunk sums down each row, then per-block bases.
// A chunk of the count matrix (MC_CHUNK consecutive blocks, all rows) is one
// contiguous run of memory; it is staged through LDS so the global reads and
// writes are coalesced and only the column walks stride.
constexpr int RS_THREADS = 256;
constexpr int RS_MAX = MC_CHUNK * (DG_MAX_BATCHES + 4);

__device__ __forceinline__ int stage_chunk(const MaskScan &a, uint32_t *s, int rows) {
  const int64_t b0 = (int64_t)blockIdx.x * MC_CHUNK;
  const int n = (int)(a.nblk - b0 < MC_CHUNK ? a.nblk - b0 : MC_CHUNK);
  const uint32_t *src = a.cnt + (size_t)b0 * rows;
  for (int i = threadIdx.x; i < n * rows; i += RS_THREADS) s[i] = src[i];
  __syncthreads();
  return n;
}

__global__ __launch_bounds__(RS_THREADS) void k_rows_chunk_sum(MaskScan a) {
  __shared__ uint32_t s[RS_MAX];
  const int rows = mc_rows(a.B);
  const int n = stage_chunk(a, s, rows);
  for (int t = threadIdx.x; t < rows; t += RS_THREADS) {
    int64_t acc = 0;
    for (int k = 0; k < n; ++k) acc += s[k * rows + t];
    a.chunk_sum[(size_t)blockIdx.x * rows + t] = acc;
  }
}

// Also stages the device error word for the caller's read-back (err_stage),
// after every kernel of the pass so far has run.
__global__ __launch_bounds__(1024) void k_rows_chunk_scan(MaskScan a) {
  const int rows = mc_rows(a.B);
  const int row = blockIdx.x;
  const int64_t nch = mc_chunks(a.nblk);
  int64_t carry = 0;
  for (int64_t c0 = 0; c0 < nch; c0 += 1024) {
    const int64_t i = c0 + threadIdx.x;
    const int64_t v = i < nch ? a.chunk_sum[(size_t)i * rows + row] : 0;
    int64_t total;
    const int64_t ex = block_excl_scan<1024>(v, &total);
    if (i < nch) a.chunk_sum[(size_t)i * rows + row] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) a.totals[row] = carry;
  if (row == 0 && threadIdx.x == 0 && a.err_stage) *a.err_stage = (int64_t)*a.err;
}

__global__ __launch_bounds__(RS_THREADS) void k_rows_apply(MaskScan a) {
  __shared__ uint32_t s[RS_MAX];
  __shared__ int64_t sb[RS_MAX];
  const int rows = mc_rows(a.B);
  const int n = stage_chunk(a, s, rows);
  for (int t = threadIdx.x; t < rows; t += RS_THREADS) {
    int64_t run = a.chunk_sum[(size_t)blockIdx.x * rows + t];
    for (int k = 0; k < n; ++k) {
      sb[k * rows + t] = run;
      run += s[k * rows + t];
    }
  }
  __syncthreads();
  int64_t *dst = a.base + (size_t)blockIdx.x * MC_CHUNK * rows;
  for (int i = threadIdx.x; i < n * rows; i += RS_THREADS) dst[i] = sb[i];
}

int mask_scan_count(MaskScan &m, hipStream_t s) {
  if (m.nblk == 0) return fill_u64(reinterpret_cast<uint64_t *>(m.totals), mc_rows(m.B), 0, s);
  const unsigned nch = (unsigned)mc_chunks(m.nblk);
  hipLaunchKernelGGL(k_mask_count, dim3((unsigned)m.nblk), dim3(MC_THREADS), 0, s, m);
  hipLaunchKernelGGL(k_rows_chunk_sum, dim3(nch), dim3(RS_THREADS), 0, s, m);
  hipLaunchKernelGGL(k_rows_chunk_scan, dim3((unsigned)mc_rows(m.B)), dim3(1024), 0, s, m);
  hipLaunchKernelGGL(k_rows_apply, dim3(nch), dim3(RS_THREADS), 0, s, m);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

// Write pass, over the compact list of non-empty words the count pass left for
// each wave (no second read of the mask).  Batch b's next rank is the block's
// base from the row scan, plus the wave's prefix within the block, plus what
// lane b has emitted so far.  Per-node outputs use ballot prefixes within a
// chunk of 64 words; the (node, batch) pairs are emitted word by word in node
// order (lane b handles bit b), so each batch's list comes out ascending.
//   PACK:  packing outputs (U, U_nc, pair offsets, pair destinations); cached
//          nodes are left out of the per-batch lists.
//   LOCAL: sampling, also recording each pair's local index in local_out.
template <bool PACK, bool LOCAL>
__global__ __launch_bounds__(MC_THREADS) void k_mask_write(MaskScan a) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const int B = a.B, rows = mc_rows(B);
  const int64_t t0 = (int64_t)blockIdx.x * MC_BLOCK_NODES + (int64_t)w * MC_TILE;
  const size_t gwi = (size_t)blockIdx.x * MC_WAVES + w;
  const uint32_t n = a.wcnt[gwi];
  if (n == 0) return;  // wave-uniform
  const uint64_t *cm = a.cw_mask + gwi * MC_TILE;
  const uint16_t *co = a.cw_off + gwi * MC_TILE;
  const int64_t *bb = a.base + (size_t)blockIdx.x * rows;
  const uint32_t *pre = a.wpre + gwi * rows;
  const int64_t run0 = lane < B ? bb[lane] + pre[lane] : 0;
  int64_t dest_b = lane < B ? a.seg_base[lane] + run0 : 0;  // next list slot of batch b
  const int64_t end_b = (!PACK && lane < B) ? a.seg_end[lane] : 0;
  int32_t local_b = 0;                                      // its local index
  if (LOCAL) local_b = lane < B ? (int32_t)(a.local_base[lane] + run0) : 0;
  int64_t run_u = 0, run_nc = 0, run_p = 0;
  if (PACK) {
    run_u = bb[row_all(B)] + pre[row_all(B)];
    run_nc = bb[row_packed(B)] + pre[row_packed(B)];
    run_p = bb[row_pairs(B)] + pre[row_pairs(B)];
  }
  const uint64_t lt = lanes_below();
  for (uint32_t c0 = 0; c0 < n; c0 += 64) {
    const uint32_t i = c0 + lane;
    uint64_t m = 0;
    uint32_t off = 0;
    if (i < n) {
      m = cm[i];
      off = co[i];
    }
    const int32_t u = (int32_t)(t0 + (off & 1023u));
    const uint64_t mnc = (PACK && (off >> 15)) ? 0ull : m;
    uint64_t anc = __ballot(mnc != 0ull);
    if (PACK) {
      const uint64_t any = __ballot(m != 0ull);
      if (m != 0ull && a.uniq_out) a.uniq_out[run_u + __popcll(any & lt)] = u;
      run_u += __popcll(any);
      const int32_t pc = __popcll(mnc);
      const int64_t pair0 = run_p + (wave_incl_sum_i32(pc) - pc);
      if (mnc != 0ull) {
        const int64_t rk = run_nc + __popcll(anc & lt);
        a.unc_ids[rk] = u;
        a.unc_off[rk] = pair0;
        a.nodeoff[u] = pair0;
      }
      run_nc += __popcll(anc);
    }
    while (anc) {
      const int l = __ffsll((long long)anc) - 1;
      anc &= ~(1ull << l);
      const uint64_t wd = (uint64_t)read_lane((int64_t)mnc, l);
      const int32_t ul = __builtin_amdgcn_readlane(u, l);
      if ((wd >> lane) & 1ull) {
        if (PACK || dest_b < end_b) a.seg_out[dest_b] = ul;
        if (PACK) a.pairdest[run_p + __popcll(wd & lt)] = dest_b;
        if (LOCAL) a.local_out[(int64_t)ul * B + lane] = local_b;
        ++dest_b;
        ++local_b;
      }
      if (PACK) run_p += __popcll(wd);
    }
  }
}

int mask_scan_write(const MaskScan &m, hipStream_t s) {
  if (m.nblk == 0) return DG_OK;
  const bool pack = m.pairdest != nullptr;
  // seg_out may be NULL only when no pair is listed (packing with every node cached)
  if ((pack && (!m.unc_ids || !m.unc_off || !m.nodeoff)) ||
      (!pack && (!m.prev || !m.seg_out || m.cache_slot || m.uniq_out)))
    return set_error(DG_EINVAL, "internal: inconsistent compaction outputs");
  const dim3 g((unsigned)m.nblk), bl(MC_THREADS);
  if (pack)
    hipLaunchKernelGGL((k_mask_write<true, false>), g, bl, 0, s, m);
  else if (m.local_out)
    hipLaunchKernelGGL((k_mask_write<false, true>), g, bl, 0, s, m);
  else
    hipLaunchKernelGGL((k_mask_write<false, false>), g, bl, 0, s, m);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

}  // namespace dg

extern "C" const char *dg_last_error(void) { return dg::g_err; }
extern "C" const char *dg_version(void) { return "libdg 0.1 (gfx950)"; }
