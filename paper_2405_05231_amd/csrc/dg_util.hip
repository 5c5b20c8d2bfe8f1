// Shared machinery of libdg: error reporting, fills, prefix scans and the
// node-major membership-mask compaction used by sampling (per-hop new-node
// lists) and packing (group unique set, per-batch packed order).
#include <stdarg.h>
#include <string.h>

#include "dg_passes.h"

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

// The same without the page-locked buffer: the copy goes to dst directly (for
// entry points that take no resources of their own).
int read_to_host_unstaged(void *dst, const void *src, size_t bytes, hipStream_t s) {
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
    DG_HIP(hipEventCreateWithFlags(&ss[dev].handoff, hipEventDisableTiming));
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

// Count pass.  One wave per tile of MC_TILE nodes, MC_ROUNDS rounds of 64.
// What is the same across the wave is kept in scalar registers: the tile base,
// the rounds that may hold a word, and for each round the lanes whose word is
// non-empty and the lanes whose node is cached; a round without a word costs a
// scalar branch only.  With touched marks a lane reads its mask word only if
// the word's 8-node line is marked.  All of a tile's mask words (then its
// prev words, then its cache slots) are requested before any is used, so a
// wave keeps up to 16 loads in flight.
//
// Per-batch counts: the tile's listed non-cached words are copied into LDS, a
// chunk of MC_CROUNDS rounds at a time, low and high halves in separate
// arrays.  Lane b then reads the halves holding bit b of four words with one
// 128-bit load (lanes 0-31 the low halves, 32-63 the high ones) and adds bit
// b mod 32 of each, so the cost per word is about 1.5 vector instructions.
//
// SAMPLE: sampling mode (prev required, no cache slots): the listed words are
// mask & ~prev, and with keep_prev the new bits are added to prev at once
// (with clear_prev the prev words read are zeroed instead).  Otherwise packing
// mode (no prev; cache_slot nullable; with clear_mask each non-zero mask word
// is zeroed once read).
constexpr int MC_CROUNDS = 4;
constexpr int MC_CWORDS = 64 * MC_CROUNDS + 4;  // + zero padding for the last read

__device__ __forceinline__ uint32_t rank_below(uint64_t set, uint32_t base) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(set >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)set, base));
}

// Waits until every vector memory load and store of the wave has completed
// (s_waitcnt vmcnt(0) in the gfx9 encoding; the other counters are left
// alone).  Placed after each branchy load phase, it tells the compiler's wait
// insertion that no load is outstanding, so no wait is placed after the stores
// that follow (a wait there would also wait for those stores).
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Eight waves per SIMD: the pass is latency-bound under load, and with the
// prev words read in two halves it fits in 64 VGPRs (a few spill to scratch);
// without the hint it takes 72 and runs seven.
template <bool SAMPLE>
__global__ __launch_bounds__(MC_THREADS) __attribute__((amdgpu_waves_per_eu(8, 8)))
void k_mask_count(MaskScan a) {
  __shared__ uint32_t s_cnt[MC_WAVES][DG_MAX_BATCHES + 4];
  __shared__ __align__(16) uint32_t s_w[MC_WAVES][2][MC_CWORDS];
  const int lane = lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int B = a.B, rows = mc_rows(B);
  const int64_t t0 = (int64_t)blockIdx.x * MC_BLOCK_NODES + (int64_t)w * MC_TILE;
  const int64_t rem = a.N - t0;  // nodes of the tile inside [0, N) (may exceed MC_TILE)

  // Touched marks: byte i of the tile's covers nodes t0 + 8i .. t0 + 8i + 7, so
  // round r's marks are the 8 bytes at 8r, and lane l's is byte l/8 of them.
  uint32_t live = 0xffffu;   // bit r: round r may hold a word (uniform)
  uint32_t lmask = 0xffffu;  // bit r: this lane's node of round r may hold one
  if (a.touched) {
    const uint64_t *f = reinterpret_cast<const uint64_t *>(a.touched + (t0 >> MC_TOUCH_SHIFT));
    const uint32_t sh = 8u * ((uint32_t)lane >> 3);
    uint32_t l = 0, lm = 0;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) {
      const uint64_t x = f[r];
      l |= (x != 0ull ? 1u : 0u) << r;
      lm |= (((x >> sh) & 0xffull) != 0ull ? 1u : 0u) << r;
    }
    live = __builtin_amdgcn_readfirstlane(l);
    lmask = lm;
  }

  uint64_t m[MC_ROUNDS];
  {
    const uint64_t *mk = a.mask + t0;
    if (rem >= MC_TILE) {
#pragma unroll
      for (int r = 0; r < MC_ROUNDS; ++r)
        m[r] = (((live >> r) & 1u) && ((lmask >> r) & 1u)) ? mk[r * 64 + lane] : 0ull;
    } else {
#pragma unroll
      for (int r = 0; r < MC_ROUNDS; ++r)
        m[r] = (((live >> r) & 1u) && ((lmask >> r) & 1u) && r * 64 + lane < rem)
                   ? mk[r * 64 + lane]
                   : 0ull;
    }
  }
  wait_vm_all();
  if (!SAMPLE && a.clear_mask) {
    uint64_t *mk = a.mask + t0;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r)
      if (m[r] != 0ull) mk[r * 64 + lane] = 0ull;
  }
  if (B < 64) {  // bits of batches outside the group are ignored
    const uint64_t keep = (1ull << B) - 1ull;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) m[r] &= keep;
  }
  if (SAMPLE && a.lines_out) {
    // member lines: round r's 8 bytes are built from its ballot (uniform) and
    // stored by lane r, 128 bytes per tile (every word was read: no marks)
    uint64_t lb = 0;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) {
      const uint64_t nz = __ballot(m[r] != 0ull);
      uint64_t v = 0;
#pragma unroll
      for (int k = 0; k < 8; ++k) v |= (((nz >> (8 * k)) & 0xffull) ? 1ull : 0ull) << (8 * k);
      if (lane == r) lb = v;
    }
    if (lane < MC_ROUNDS)
      reinterpret_cast<uint64_t *>(a.lines_out + (t0 >> MC_TOUCH_SHIFT))[lane] = lb;
  }
  uint64_t any[MC_ROUNDS];  // lanes of round r with a word to list (uniform)
#pragma unroll
  for (int r = 0; r < MC_ROUNDS; ++r) any[r] = ((live >> r) & 1u) ? __ballot(m[r] != 0ull) : 0ull;

  uint64_t cmask[MC_ROUNDS];  // lanes of round r whose node is cached (uniform)
#pragma unroll
  for (int r = 0; r < MC_ROUNDS; ++r) cmask[r] = 0ull;
  if (SAMPLE) {
    // prev's lines: bit r of plm says this lane's line in round r holds a prev
    // bit; the prev word is read only then (round r's marks are the 8 bytes at
    // 8r, and lane l's is byte l/8 of them, as for the touched marks)
    uint32_t plm = 0xffffu;
    if (a.plines) {
      const uint64_t *f = reinterpret_cast<const uint64_t *>(a.plines + (t0 >> MC_TOUCH_SHIFT));
      const uint32_t sh = 8u * ((uint32_t)lane >> 3);
      uint32_t lm = 0;
#pragma unroll
      for (int r = 0; r < MC_ROUNDS; ++r)
        lm |= (((f[r] >> sh) & 0xffull) != 0ull ? 1u : 0u) << r;
      plm = lm;
      if (a.clear_prev) {  // the marks go with the prev words they describe
        uint64_t *fw = reinterpret_cast<uint64_t *>(a.plines + (t0 >> MC_TOUCH_SHIFT));
        const uint64_t mine = lane < MC_ROUNDS ? f[lane] : 0ull;
        if (mine != 0ull) fw[lane] = 0ull;
      }
    }
    // prev words in two halves of the rounds: half the registers (so more
    // waves per SIMD) for one more round trip
    uint64_t *pv = a.prev + t0;
    constexpr int H = MC_ROUNDS / 2;
#pragma unroll
    for (int h0 = 0; h0 < MC_ROUNDS; h0 += H) {
      uint64_t p[H];
#pragma unroll
      for (int q = 0; q < H; ++q) {
        const int r = h0 + q;
        p[q] = (any[r] && m[r] != 0ull && ((plm >> r) & 1u)) ? pv[r * 64 + lane] : 0ull;
      }
      wait_vm_all();
#pragma unroll
      for (int q = 0; q < H; ++q) {
        const int r = h0 + q;
        if (!any[r]) continue;
        const uint64_t nw = m[r] & ~p[q];
        if (a.keep_prev && nw != 0ull) pv[r * 64 + lane] = p[q] | nw;
        if (a.clear_prev && p[q] != 0ull) pv[r * 64 + lane] = 0ull;
        m[r] = nw;
        any[r] = __ballot(nw != 0ull);
        if (a.keep_prev && a.plines) {  // the lines of this hop's new words
          const uint32_t sh = 8u * (uint32_t)lane;
          if (lane < 8 && ((any[r] >> sh) & 0xffull) != 0ull)
            a.plines[(t0 >> MC_TOUCH_SHIFT) + r * 8 + lane] = 1;
        }
      }
    }
  } else if (a.cache_slot) {
    const int32_t *cs = a.cache_slot + t0;
    int32_t sl[MC_ROUNDS];
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) sl[r] = (any[r] && m[r] != 0ull) ? cs[r * 64 + lane] : -1;
    wait_vm_all();
    uint64_t bad = 0;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) {
      if (!any[r]) continue;
      bad |= __ballot(sl[r] < -1);
      cmask[r] = __ballot(sl[r] >= 0);
    }
    if (bad && lane == 0) atomicOr(a.err, ERR_CACHE_SLOT);
  }

  // List the non-empty words (global, for the write pass) and count.
  const size_t gw = ((size_t)blockIdx.x * MC_WAVES + w) * MC_TILE;
  uint32_t *lo_w = s_w[w][0], *hi_w = s_w[w][1];
  const uint4 *src4 = reinterpret_cast<const uint4 *>(lane < 32 ? lo_w : hi_w);
  const uint32_t sh = (uint32_t)lane & 31u;
  uint32_t run = 0, cu = 0, cnc = 0;  // uniform
  uint32_t al = 0, pl = 0, mine = 0;  // this lane's pairs (all, non-cached), batch `lane`
#pragma unroll
  for (int c = 0; c < MC_ROUNDS; c += MC_CROUNDS) {
    uint32_t k = 0;  // non-cached words of the chunk (uniform)
#pragma unroll
    for (int r = c; r < c + MC_CROUNDS; ++r) {
      const uint64_t an = any[r];
      if (!an) continue;
      const uint64_t anc = an & ~cmask[r];
      const uint32_t pc = (uint32_t)__popcll(m[r]);
      al += pc;
      if (m[r] != 0ull) {
        const bool cached = (cmask[r] >> lane) & 1ull;
        const size_t at = gw + rank_below(an, run);
        a.cw_mask[at] = m[r];
        a.cw_off[at] = (uint16_t)((r * 64 + lane) | ((int)cached << 15));
        if (!cached) {
          pl += pc;
          const uint32_t j = rank_below(anc, k);
          lo_w[j] = (uint32_t)m[r];
          hi_w[j] = (uint32_t)(m[r] >> 32);
        }
      }
      run += (uint32_t)__popcll(an);
      cu += (uint32_t)__popcll(an);
      cnc += (uint32_t)__popcll(anc);
      k += (uint32_t)__popcll(anc);
    }
    if (k == 0) continue;
    if (lane < 4) {  // zeros after the last word: the final 128-bit read may pass it
      lo_w[k + lane] = 0u;
      hi_w[k + lane] = 0u;
    }
    // LDS operations of one wave complete in order, so these reads see the
    // stores above and the next chunk's stores follow them.
    __builtin_amdgcn_wave_barrier();
    for (uint32_t i = 0; i < k; i += 4) {
      const uint4 v = src4[i >> 2];
      mine += __builtin_amdgcn_ubfe(v.x, sh, 1) + __builtin_amdgcn_ubfe(v.y, sh, 1);
      mine += __builtin_amdgcn_ubfe(v.z, sh, 1) + __builtin_amdgcn_ubfe(v.w, sh, 1);
    }
    __builtin_amdgcn_wave_barrier();
  }
  if (lane == 0) a.wcnt[(size_t)blockIdx.x * MC_WAVES + w] = run;
  const uint32_t call = (uint32_t)__ockl_wfred_add_i32((int32_t)al);
  const uint32_t cp = SAMPLE ? call : (uint32_t)__ockl_wfred_add_i32((int32_t)pl);

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

// Member lines from the mask alone (for sweeps that did not read every word):
// byte i = 1 iff one of words 8i .. 8i+7 (below N) has a bit of batches < B.
__global__ __launch_bounds__(256) void k_member_lines(const uint64_t *mask, int64_t N, int B,
                                                      int64_t nbytes, uint8_t *out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= nbytes) return;
  const uint64_t keep = B < 64 ? (1ull << B) - 1ull : ~0ull;
  uint64_t any = 0;
  const int64_t u0 = i << MC_TOUCH_SHIFT;
  for (int k = 0; k < (1 << MC_TOUCH_SHIFT); ++k)
    if (u0 + k < N) any |= mask[u0 + k] & keep;
  out[i] = any ? 1 : 0;
}

int member_lines_pass(const uint64_t *mask, int64_t N, int B, uint8_t *out, hipStream_t s) {
  const int64_t nbytes = mc_touch_bytes(N);
  if (nbytes == 0) return DG_OK;
  hipLaunchKernelGGL(k_member_lines, dim3((unsigned)((nbytes + 255) / 256)), dim3(256), 0, s,
                     mask, N, B, nbytes, out);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

int mask_scan_count(MaskScan &m, hipStream_t s) {
  if (m.nblk == 0) return fill_u64(reinterpret_cast<uint64_t *>(m.totals), mc_rows(m.B), 0, s);
  if ((m.prev && (m.cache_slot || m.clear_mask)) || (m.keep_prev && m.clear_prev) ||
      (!m.prev && (m.keep_prev || m.clear_prev || m.lines_out)) || (m.lines_out && m.touched))
    return set_error(DG_EINVAL, "internal: inconsistent count-pass mode");
  if (m.prev)
    hipLaunchKernelGGL(k_mask_count<true>, dim3((unsigned)m.nblk), dim3(MC_THREADS), 0, s, m);
  else
    hipLaunchKernelGGL(k_mask_count<false>, dim3((unsigned)m.nblk), dim3(MC_THREADS), 0, s, m);
  DG_HIP(hipGetLastError());
  return mask_scan_rows(m, s);
}

int mask_scan_rows(MaskScan &m, hipStream_t s) {
  if (m.nblk == 0) return fill_u64(reinterpret_cast<uint64_t *>(m.totals), mc_rows(m.B), 0, s);
  const unsigned nch = (unsigned)mc_chunks(m.nblk);
  hipLaunchKernelGGL(k_rows_chunk_sum, dim3(nch), dim3(RS_THREADS), 0, s, m);
  hipLaunchKernelGGL(k_rows_chunk_scan, dim3((unsigned)mc_rows(m.B)), dim3(1024), 0, s, m);
  hipLaunchKernelGGL(k_rows_apply, dim3(nch), dim3(RS_THREADS), 0, s, m);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

// 64 x 64 bit transpose across the wave: lane i holds row i (bit j is entry
// (i, j)); on return lane j holds column j (bit i is entry (i, j)).  Each of
// the six block-swap stages exchanges bit s of the row index with bit s of the
// column index between lanes i and i ^ s.  The stage across the wave halves
// moves 32-bit halves by a lane shuffle; the five within each half work on
// the 32-bit halves of the rows, which those stages never mix, and take the
// partner's value by DPP (s = 1, 2 within quads, 4 and 8 within rows of 16
// lanes) or by ds_swizzle (s = 16).
template <int S>
__device__ __forceinline__ uint32_t xor_partner(uint32_t v, int lane) {
  if constexpr (S == 1) {  // quad_perm [1, 0, 3, 2]
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xb1, 0xf, 0xf, false);
  } else if constexpr (S == 2) {  // quad_perm [2, 3, 0, 1]
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4e, 0xf, 0xf, false);
  } else if constexpr (S == 4 || S == 8) {
    // row_shl:S (lane i reads lane i + S) for the lanes with bit S clear,
    // row_shr:S (lane i reads lane i - S) for the others; both stay in the row
    const uint32_t up = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x100 | S, 0xf, 0xf, false);
    const uint32_t dn = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x110 | S, 0xf, 0xf, false);
    return (lane & S) ? dn : up;
  } else {
    static_assert(S == 16, "xor within 32 lanes");
    return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, (S << 10) | 0x1f);
  }
}
template <int S>
__device__ __forceinline__ void transpose_stage(uint32_t &lo, uint32_t &hi, int lane) {
  // positions whose bit S is clear, in each 32-bit half
  constexpr uint32_t M0 = S == 16 ? 0x0000ffffu : S == 8 ? 0x00ff00ffu : S == 4 ? 0x0f0f0f0fu
                        : S == 2 ? 0x33333333u : 0x55555555u;
  const bool low = (lane & S) == 0;
  const uint32_t plo = xor_partner<S>(lo, lane), phi = xor_partner<S>(hi, lane);
  // low lane: keeps its M0 positions, takes the partner's M0 positions moved up
  // by S; high lane: keeps its other positions, takes the partner's moved down
  const uint32_t keep = low ? M0 : ~M0;
  const uint32_t xlo = low ? plo << S : plo >> S;
  const uint32_t xhi = low ? phi << S : phi >> S;
  lo = (lo & keep) | (xlo & ~keep);
  hi = (hi & keep) | (xhi & ~keep);
}
__device__ __forceinline__ uint64_t wave_transpose64(uint64_t r) {
  const int lane = lane_id();
  uint32_t lo = (uint32_t)r, hi = (uint32_t)(r >> 32);
  {  // bit 5: the low lane of a pair takes its partner's low half as its high
     // half, the high lane its partner's high half as its low half
    const bool low = (lane & 32) == 0;
    const uint32_t got = (uint32_t)__shfl_xor((int)(low ? hi : lo), 32, 64);
    if (low) hi = got; else lo = got;
  }
  transpose_stage<16>(lo, hi, lane);
  transpose_stage<8>(lo, hi, lane);
  transpose_stage<4>(lo, hi, lane);
  transpose_stage<2>(lo, hi, lane);
  transpose_stage<1>(lo, hi, lane);
  return ((uint64_t)hi << 32) | lo;
}

// Write pass, over the compact list of non-empty words the count pass left for
// each wave (no second read of the mask).  Batch b's next rank is the block's
// base from the row scan, plus the wave's prefix within the block, plus what
// lane b has emitted so far.  Per-node outputs use ballot prefixes within a
// chunk of 64 words.  For the (node, batch) pairs the chunk's words are
// transposed, so that lane b holds the set of the chunk's words with bit b,
// and lane b walks that set in node order (the words' node IDs, cache slots
// and pair offsets staged in LDS): each batch's list comes out ascending, and
// a lane's walk is as long as its batch's share of the chunk.
//   PACK:  packing outputs (U, U_nc, pair offsets, pair destinations); cached
//          nodes are left out of the per-batch lists.
//   LOCAL: sampling, also recording each pair's local index in local_out.
// Sampling with loc_out also writes each listed pair's address-table entry,
// at the index of its list slot: the entry of a cached node is final, the
// others are left DG_LOC_PENDING for packing.  Each lane loads the cache slot
// of its own word before the pairs are emitted.
template <bool PACK, bool LOCAL>
__global__ __launch_bounds__(MC_THREADS) void k_mask_write(MaskScan a) {
  // per word of the chunk: first pair (packing, from run_p) << 10 | node
  // offset in the tile, cache slot, listed bits (packing)
  __shared__ int4 s_word[MC_WAVES][64];
  const int lane = lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int B = a.B, rows = mc_rows(B);
  // Neighbouring blocks append to the same stretch of every batch's list: run
  // them on one XCD, so that lines shared between them merge in its L2.
  const uint32_t blk = xcd_block(blockIdx.x, gridDim.x);
  const int64_t t0 = (int64_t)blk * MC_BLOCK_NODES + (int64_t)w * MC_TILE;
  const size_t gwi = (size_t)blk * MC_WAVES + w;
  const uint64_t *cm = a.cw_mask + gwi * MC_TILE;
  const uint16_t *co = a.cw_off + gwi * MC_TILE;
  const int64_t *bb = a.base + (size_t)blk * rows;
  const uint32_t *pre = a.wpre + gwi * rows;
  // The count, the bases and the first chunk are requested together: the
  // chunk's 64 entries lie inside the wave's part of the compact list
  // whatever the count.
  const uint32_t n = a.wcnt[gwi];
  uint64_t m = cm[lane];
  uint32_t off = co[lane];
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
  wait_vm_all();
  if (n == 0) return;  // wave-uniform
  const uint64_t lt = lanes_below();
  for (uint32_t c0 = 0; c0 < n; c0 += 64) {
    const uint32_t i = c0 + lane;
    if (c0 > 0) {
      if (i < n) {
        m = cm[i];
        off = co[i];
      }
      wait_vm_all();  // as in the fused write pass
    }
    if (i >= n) {
      m = 0;
      off = 0;
    }
    const int32_t u = (int32_t)(t0 + (off & 1023u));
    int32_t sl = -1;  // sampling with loc_out: this lane's node's cache slot
    if (!PACK && a.loc_out && i < n) {
      sl = a.loc_slot[u];
      if (sl < -1) atomicOr(a.err, ERR_CACHE_SLOT);
    }
    const uint64_t mnc = (PACK && (off >> 15)) ? 0ull : m;
    const uint64_t anc = __ballot(mnc != 0ull);
    int32_t p0 = 0, incl = 0;  // packing: the word's first pair, from run_p
    if (PACK) {
      const uint64_t any = __ballot(m != 0ull);
      if (m != 0ull && a.uniq_out) a.uniq_out[run_u + __popcll(any & lt)] = u;
      run_u += __popcll(any);
      const int32_t pc = __popcll(mnc);
      incl = wave_incl_sum_i32(pc);
      p0 = incl - pc;
      if (mnc != 0ull) {
        const int64_t rk = run_nc + __popcll(anc & lt);
        a.unc_ids[rk] = u;
        a.unc_off[rk] = run_p + p0;
        a.nodeoff[u] = run_p + p0;
      }
      run_nc += __popcll(anc);
    }
    if (!anc) continue;  // uniform
    uint64_t todo = wave_transpose64(mnc);  // lane b: the chunk's words with bit b
    s_word[w][lane] = int4{(p0 << 10) | (int32_t)(off & 1023u), sl, (int32_t)(uint32_t)mnc,
                           (int32_t)(uint32_t)(mnc >> 32)};
    // LDS operations of one wave complete in order: the reads below see these
    // stores, and the next chunk's stores follow this chunk's reads.
    __builtin_amdgcn_wave_barrier();
    int k = todo ? __builtin_ctzll(todo) : 0;
    int4 e = s_word[w][k];
    while (todo) {
      todo &= todo - 1ull;
      const int kn = todo ? __builtin_ctzll(todo) : k;
      const int4 en = s_word[w][kn];  // the next word's entry, requested ahead
      const int32_t uk = (int32_t)(t0 + (e.x & 1023));
      if (PACK || dest_b < end_b) a.seg_out[dest_b] = uk;
      if (!PACK && a.loc_out && dest_b < end_b)
        a.loc_out[dest_b] = e.y >= 0 ? -(e.y + 1) : (int32_t)DG_LOC_PENDING;
      if (PACK) {
        const uint64_t mk = ((uint64_t)(uint32_t)e.w << 32) | (uint32_t)e.z;
        a.pairdest[run_p + (e.x >> 10) + __popcll(mk & lt)] = dest_b;
      }
      if (LOCAL) a.local_out[(int64_t)uk * B + lane] = local_b;
      ++dest_b;
      ++local_b;
      e = en;
    }
    __builtin_amdgcn_wave_barrier();
    if (PACK) run_p += __builtin_amdgcn_readlane(incl, 63);
  }
}

int mask_scan_write(const MaskScan &m, hipStream_t s) {
  if (m.nblk == 0) return DG_OK;
  const bool pack = m.pairdest != nullptr;
  // seg_out may be NULL only when no pair is listed (packing with every node cached)
  if ((pack && (!m.unc_ids || !m.unc_off || !m.nodeoff)) ||
      (!pack && (!m.prev || !m.seg_out || m.cache_slot || m.uniq_out)) ||
      (pack && m.loc_out) || (!m.loc_out != !m.loc_slot))
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

// ---------------------------------------------------------------- fused compaction
// Adds bit `lane & 31` of the low (lanes < 32) or high (lanes >= 32) halves of
// the k words staged in lo/hi to `mine` (batch `lane`'s count), four words
// per 128-bit LDS read.  The staging areas hold MC_CWORDS entries.
__device__ __forceinline__ void lds_count(uint32_t k, uint32_t *lo, uint32_t *hi, int lane,
                                          uint32_t &mine) {
  if (k == 0) return;  // uniform
  if (lane < 4) {      // zeros after the last word: the final 128-bit read may pass it
    lo[k + lane] = 0u;
    hi[k + lane] = 0u;
  }
  // LDS operations of one wave complete in order, so these reads see the
  // stores above and later stores follow them.
  __builtin_amdgcn_wave_barrier();
  const uint4 *src = reinterpret_cast<const uint4 *>(lane < 32 ? lo : hi);
  const uint32_t sh = (uint32_t)lane & 31u;
  for (uint32_t i = 0; i < k; i += 4) {
    const uint4 v = src[i >> 2];
    mine += __builtin_amdgcn_ubfe(v.x, sh, 1) + __builtin_amdgcn_ubfe(v.y, sh, 1);
    mine += __builtin_amdgcn_ubfe(v.z, sh, 1) + __builtin_amdgcn_ubfe(v.w, sh, 1);
  }
  __builtin_amdgcn_wave_barrier();
}

// Fused count pass (FuseScan).  Every word is read (no touched marks).  The
// tile is taken in four parts of four rounds, so that a part's mask words,
// prev words and cache slots are in registers together without spilling; the
// next part's mask words are requested together with this part's prev words
// and cache slots, so a part costs one round trip.  Per-batch counts, a part
// at a time: the part's words with new bits are staged in one LDS area and its
// non-cached words in another, and lane b counts bit b of each.
constexpr int FC_PART = MC_ROUNDS / 4;

// It runs eight waves per SIMD without a hint (54 VGPRs); a hint of eight
// waves caps its scalar registers at 80 and spills 20 of them into vector
// lanes (about 150 more vector instructions per wave).
__global__ __launch_bounds__(MC_THREADS) void k_fuse_count(FuseScan a) {
  __shared__ uint32_t s_cs[MC_WAVES][DG_MAX_BATCHES + 4];
  __shared__ uint32_t s_cp[MC_WAVES][DG_MAX_BATCHES + 4];
  __shared__ __align__(16) uint32_t s_w[MC_WAVES][4][MC_CWORDS];
  const int lane = lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int B = a.B, rows = mc_rows(B);
  const int64_t t0 = (int64_t)blockIdx.x * MC_BLOCK_NODES + (int64_t)w * MC_TILE;
  const int64_t rem = a.N - t0;  // nodes of the tile inside [0, N) (may exceed MC_TILE)
  const uint64_t keep = B < 64 ? (1ull << B) - 1ull : ~0ull;
  const size_t gw = ((size_t)blockIdx.x * MC_WAVES + w) * MC_TILE;
  uint32_t *ns_lo = s_w[w][0], *ns_hi = s_w[w][1];  // words with new bits
  uint32_t *np_lo = s_w[w][2], *np_hi = s_w[w][3];  // words of non-cached nodes
  uint64_t *mk = a.mask + t0;
  uint64_t *pv = a.prev + t0;
  const int32_t *cs = a.cache_slot + t0;
  uint32_t run = 0, cu = 0, cnc = 0, cnew = 0;  // uniform: listed, U, U_nc, new words
  uint32_t al = 0, pl = 0, nl = 0;  // this lane's word: all, non-cached, new pairs
  uint32_t mine_s = 0, mine_p = 0;  // batch `lane`: new pairs, non-cached pairs
  uint64_t bad = 0;
  // Mask words are loaded unconditionally (a node past N reads the last word,
  // and its value is dropped): no branch between the loads of a part.
  auto load_part = [&](int h0, uint64_t (&m)[FC_PART]) {
#pragma unroll
    for (int q = 0; q < FC_PART; ++q) {
      const int64_t r = (int64_t)(h0 + q) * 64 + lane;
      m[q] = a.mask[r < rem ? t0 + r : a.N - 1];
    }
#pragma unroll
    for (int q = 0; q < FC_PART; ++q)
      if ((int64_t)(h0 + q) * 64 + lane >= rem) m[q] = 0ull;
  };
  // prev's lines (bit r: this lane's line in round r holds a prev bit; the
  // prev word is read only then), zeroed with the prev words
  uint32_t plm = 0xffffu;
  if (a.plines) {
    const uint64_t *f = reinterpret_cast<const uint64_t *>(a.plines + (t0 >> MC_TOUCH_SHIFT));
    const uint32_t sh = 8u * ((uint32_t)lane >> 3);
    uint32_t lm = 0;
#pragma unroll
    for (int r = 0; r < MC_ROUNDS; ++r) lm |= (((f[r] >> sh) & 0xffull) != 0ull ? 1u : 0u) << r;
    plm = lm;
    if (a.clear_prev) {
      uint64_t *fw = reinterpret_cast<uint64_t *>(a.plines + (t0 >> MC_TOUCH_SHIFT));
      const uint64_t mine = lane < MC_ROUNDS ? f[lane] : 0ull;
      if (mine != 0ull) fw[lane] = 0ull;
    }
  }
  uint64_t m[FC_PART];
  load_part(0, m);
  wait_vm_all();
#pragma unroll
  for (int h0 = 0; h0 < MC_ROUNDS; h0 += FC_PART) {
    uint64_t any[FC_PART];  // lanes of round q with a word (uniform)
    uint64_t nw[FC_PART];
    int32_t sl[FC_PART];
#pragma unroll
    for (int q = 0; q < FC_PART; ++q) {
      const bool has = (m[q] & keep) != 0ull;
      any[q] = __ballot(has);
      nw[q] = (has && ((plm >> (h0 + q)) & 1u)) ? pv[(h0 + q) * 64 + lane] : 0ull;
      sl[q] = has ? cs[(h0 + q) * 64 + lane] : -1;
    }
    uint64_t mn[FC_PART];  // the next part's mask words
    if (h0 + FC_PART < MC_ROUNDS) load_part(h0 + FC_PART, mn);
    wait_vm_all();
    // The cached lanes of each round, and each listed word's slot at its place
    // in the compact list (so that the slots need no registers further on).
    uint64_t cmask[FC_PART];  // cached lanes of round q (uniform)
    {
      uint32_t at0 = run;
#pragma unroll
      for (int q = 0; q < FC_PART; ++q) {
        cmask[q] = 0ull;
        if (!any[q]) continue;
        bad |= __ballot(sl[q] < -1);
        cmask[q] = __ballot(sl[q] >= 0);
        if ((m[q] & keep) != 0ull) a.cw_slot[gw + rank_below(any[q], at0)] = sl[q];
        at0 += (uint32_t)__popcll(any[q]);
      }
    }
#pragma unroll
    for (int c = 0; c < FC_PART; c += MC_CROUNDS) {
      uint32_t ks = 0, kp = 0;  // staged new / non-cached words of the chunk (uniform)
#pragma unroll
      for (int q = c; q < c + MC_CROUNDS; ++q) {
        const int r = h0 + q;
        if (m[q] != 0ull) mk[r * 64 + lane] = 0ull;  // packing consumes the word
        const uint64_t p = nw[q];
        if (a.clear_prev && p != 0ull) pv[r * 64 + lane] = 0ull;
        const uint64_t mq = m[q] & keep;
        const uint64_t nq = mq & ~p;
        const uint64_t an = any[q];
        if (!an) continue;
        const uint64_t cmq = cmask[q];
        const uint64_t anw = __ballot(nq != 0ull);  // lanes with new bits (uniform)
        const uint64_t anc = an & ~cmq;
        if (mq != 0ull) {
          const bool cached = (cmq >> lane) & 1ull;
          const size_t at = gw + rank_below(an, run);
          a.cw_mask[at] = mq;
          a.cw_new[at] = nq;
          a.cw_off[at] = (uint16_t)((r * 64 + lane) | ((int)cached << 15));
          const uint32_t pc = (uint32_t)__popcll(mq);
          al += pc;
          if (nq != 0ull) {
            nl += (uint32_t)__popcll(nq);
            const uint32_t j = rank_below(anw, ks);
            ns_lo[j] = (uint32_t)nq;
            ns_hi[j] = (uint32_t)(nq >> 32);
          }
          if (!cached) {
            pl += pc;
            const uint32_t j = rank_below(anc, kp);
            np_lo[j] = (uint32_t)mq;
            np_hi[j] = (uint32_t)(mq >> 32);
          }
        }
        run += (uint32_t)__popcll(an);
        cu += (uint32_t)__popcll(an);
        cnc += (uint32_t)__popcll(anc);
        cnew += (uint32_t)__popcll(anw);
        ks += (uint32_t)__popcll(anw);
        kp += (uint32_t)__popcll(anc);
      }
      lds_count(ks, ns_lo, ns_hi, lane, mine_s);
      lds_count(kp, np_lo, np_hi, lane, mine_p);
    }
    if (h0 + FC_PART < MC_ROUNDS) {
#pragma unroll
      for (int q = 0; q < FC_PART; ++q) m[q] = mn[q];
    }
  }
  if (bad && lane == 0) atomicOr(a.err, ERR_CACHE_SLOT);
  const size_t gwi = (size_t)blockIdx.x * MC_WAVES + w;
  if (lane == 0) a.wcnt[gwi] = run;
  const uint32_t sum_all = (uint32_t)__ockl_wfred_add_i32((int32_t)al);
  const uint32_t sum_nc = (uint32_t)__ockl_wfred_add_i32((int32_t)pl);
  const uint32_t sum_new = (uint32_t)__ockl_wfred_add_i32((int32_t)nl);
  if (lane < B) {
    s_cs[w][lane] = mine_s;
    s_cp[w][lane] = mine_p;
  }
  if (lane == 0) {
    s_cs[w][row_all(B)] = cnew;
    s_cs[w][row_packed(B)] = cnew;
    s_cs[w][row_pairs(B)] = sum_new;
    s_cs[w][row_all_pairs(B)] = sum_new;
    s_cp[w][row_all(B)] = cu;
    s_cp[w][row_packed(B)] = cnc;
    s_cp[w][row_pairs(B)] = sum_nc;
    s_cp[w][row_all_pairs(B)] = sum_all;
  }
  __syncthreads();
  uint32_t *pre_s = a.wpre_s + (size_t)blockIdx.x * MC_WAVES * rows;
  uint32_t *pre_p = a.wpre_p + (size_t)blockIdx.x * MC_WAVES * rows;
  for (int i = threadIdx.x; i < 2 * rows; i += MC_THREADS) {
    const bool sv = i < rows;
    const int row = sv ? i : i - rows;
    uint32_t *pre = sv ? pre_s : pre_p;
    uint32_t v = 0;
#pragma unroll
    for (int j = 0; j < MC_WAVES; ++j) {
      pre[j * rows + row] = v;
      v += sv ? s_cs[j][row] : s_cp[j][row];
    }
    (sv ? a.cnt_s : a.cnt_p)[(size_t)blockIdx.x * rows + row] = v;
  }
}

// packed_ptr from the p view's per-batch totals.
__global__ void k_fuse_ptr(const int64_t *totals, int B, int64_t *packed_ptr) {
  if (threadIdx.x == 0) {
    int64_t run = 0;
    packed_ptr[0] = 0;
    for (int b = 0; b < B; ++b) {
      run += totals[b];
      packed_ptr[b + 1] = run;
    }
  }
}

// Fused write pass (FuseScan), over the compact list, 64 words at a time.
// Per-node outputs (U, U_nc, pair offsets) by ballot prefixes within the
// chunk, as in packing's write pass.  Then lane b takes batch b's pairs: the
// chunk's new bits and non-cached bits are transposed, so that lane b holds
// the set of the chunk's words with bit b, and walks that set in list order
// (the words' node IDs, cache slots and pair offsets staged in LDS).  A new
// pair goes to batch b's segment (with its address-table entry when the node
// is cached, and its local index when local_out is given), a non-cached pair
// to P_b with its destination and list slot.  A lane's walk is as long as its
// batch's share of the chunk, a few words where the chunk's nodes are cold,
// instead of one step per word for every lane.  Blocks run in XCD-contiguous
// order, as in the other write pass.
__global__ __launch_bounds__(MC_THREADS) void k_fuse_write(FuseScan a) {
  // per word of the chunk: first pair (from run_p) << 10 | node offset in the
  // tile, cache slot, non-cached bits
  __shared__ int4 s_word[MC_WAVES][64];
  const int lane = lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int B = a.B, rows = mc_rows(B);
  const uint32_t blk = xcd_block(blockIdx.x, gridDim.x);
  const int64_t t0 = (int64_t)blk * MC_BLOCK_NODES + (int64_t)w * MC_TILE;
  const size_t gwi = (size_t)blk * MC_WAVES + w;
  const uint64_t *cm = a.cw_mask + gwi * MC_TILE;
  const uint64_t *cn = a.cw_new + gwi * MC_TILE;
  const uint16_t *co = a.cw_off + gwi * MC_TILE;
  const int32_t *csl = a.cw_slot + gwi * MC_TILE;
  const int64_t *bs = a.base_s + (size_t)blk * rows;
  const int64_t *bp = a.base_p + (size_t)blk * rows;
  const uint32_t *ps = a.wpre_s + gwi * rows;
  const uint32_t *pp = a.wpre_p + gwi * rows;
  // The count, the bases and the first chunk are requested together: the
  // chunk's 64 entries lie inside the wave's part of the compact list
  // whatever the count.
  const uint32_t n = a.wcnt[gwi];
  uint64_t m = cm[lane], nw = cn[lane];
  uint32_t off = co[lane];
  int32_t sl = csl[lane];  // the node's cache slot (for a cached node's new pairs)
  // batch `lane`: the next slot of its segment (dest_b; li within the batch's
  // node_cap entries) and the next row of its chunk of P
  int64_t dest_b = 0, pd_b = 0;
  int32_t li = 0;
  if (lane < B) {
    dest_b = a.seg_base[lane] + bs[lane] + ps[lane];
    li = (int32_t)(dest_b - (int64_t)lane * a.node_cap);
    pd_b = a.packed_ptr[lane] + bp[lane] + pp[lane];
  }
  int64_t run_u = bp[row_all(B)] + pp[row_all(B)];
  int64_t run_nc = bp[row_packed(B)] + pp[row_packed(B)];
  int64_t run_p = bp[row_pairs(B)] + pp[row_pairs(B)];
  wait_vm_all();
  if (n == 0) return;  // wave-uniform
  const uint64_t lt = lanes_below();
  for (uint32_t c0 = 0; c0 < n; c0 += 64) {
    const uint32_t i = c0 + lane;
    if (c0 > 0) {
      if (i < n) {
        m = cm[i];
        nw = cn[i];
        off = co[i];
        sl = csl[i];
      }
      // The chunk's loads have landed before its first store: the loads and
      // stores share one counter, so a wait placed after the stores below
      // (the compiler's choice for values loaded in the loop) would also wait
      // for every store.
      wait_vm_all();
    }
    if (i >= n) {
      m = nw = 0;
      off = 0;
      sl = -1;
    }
    const int32_t u = (int32_t)(t0 + (off & 1023u));
    const bool cached = (off >> 15) & 1u;
    const uint64_t mnc = cached ? 0ull : m;
    const uint64_t any = __ballot(m != 0ull);
    if (m != 0ull && a.uniq_out) {
      const int64_t at = run_u + __popcll(any & lt);
      if (at < a.unique_cap) a.uniq_out[at] = u;
    }
    run_u += __popcll(any);
    const uint64_t anc = __ballot(mnc != 0ull);
    const int32_t pc = __popcll(mnc);
    const int32_t incl = wave_incl_sum_i32(pc);
    const int32_t p0 = incl - pc;  // the word's first pair, from run_p
    if (mnc != 0ull) {
      const int64_t rk = run_nc + __popcll(anc & lt);
      if (rk < a.unc_cap) {
        a.unc_ids[rk] = u;
        a.unc_off[rk] = run_p + p0;
      }
      if (a.nodeoff) a.nodeoff[u] = run_p + p0;
    }
    run_nc += __popcll(anc);
    const bool has_new = __ballot(nw != 0ull) != 0ull;  // uniform
    const uint64_t tn = has_new ? wave_transpose64(nw) : 0ull;  // lane b: words with new bit b
    const uint64_t tp = anc ? wave_transpose64(mnc) : 0ull;      // lane b: words with non-cached bit b
    s_word[w][lane] = int4{(p0 << 10) | (int32_t)(off & 1023u), sl, (int32_t)(uint32_t)mnc,
                           (int32_t)(uint32_t)(mnc >> 32)};
    // LDS operations of one wave complete in order: the reads below see these
    // stores, and the next chunk's stores follow this chunk's reads.
    __builtin_amdgcn_wave_barrier();
    uint64_t todo = tn | tp;
    int k = todo ? __builtin_ctzll(todo) : 0;
    int4 e = s_word[w][k];
    while (todo) {
      todo &= todo - 1ull;
      const int kn = todo ? __builtin_ctzll(todo) : k;
      const int4 en = s_word[w][kn];  // the next word's entry, requested ahead
      const int32_t uk = (int32_t)(t0 + (e.x & 1023));
      const int32_t slot = li;
      const bool is_new = (tn >> k) & 1ull;
      if (is_new) {
        if (li < a.node_cap) {
          a.seg_out[dest_b] = uk;
          if (e.y >= 0) a.loc_out[dest_b] = -(e.y + 1);
          if (a.local_out) a.local_out[(int64_t)uk * B + lane] = li;
        }
        ++dest_b;
        ++li;
      }
      if ((tp >> k) & 1ull) {
        if (pd_b < a.packed_cap)
          a.pinfo[pd_b] = ((uint64_t)(uint32_t)(is_new ? slot : -1) << 32) | (uint32_t)uk;
        const uint64_t mk = ((uint64_t)(uint32_t)e.w << 32) | (uint32_t)e.z;
        const int64_t q = run_p + (e.x >> 10) + __popcll(mk & lt);
        if (q < a.pair_cap) a.pairdest[q] = pd_b;
        ++pd_b;
      }
      k = kn;
      e = en;
    }
    __builtin_amdgcn_wave_barrier();
    run_p += __builtin_amdgcn_readlane(incl, 63);
  }
}

int fuse_scan_count(const FuseScan &f, MaskScan &vs, MaskScan &vp, hipStream_t s) {
  if (!f.mask || !f.prev || !f.cache_slot || !f.cw_slot || vs.nblk != f.nblk || vp.nblk != f.nblk ||
      vs.B != f.B || vp.B != f.B)
    return set_error(DG_EINVAL, "internal: inconsistent fused count pass");
  if (f.nblk > 0) {
    hipLaunchKernelGGL(k_fuse_count, dim3((unsigned)f.nblk), dim3(MC_THREADS), 0, s, f);
    DG_HIP(hipGetLastError());
  }
  int rc;
  if ((rc = mask_scan_rows(vs, s))) return rc;
  return mask_scan_rows(vp, s);
}

int fuse_scan_write(const FuseScan &f, const int64_t *totals_p, int64_t *packed_ptr,
                    hipStream_t s) {
  if (!f.seg_out || !f.loc_out || !f.unc_ids || !f.unc_off || !f.pairdest || !f.cw_slot ||
      (f.packed_cap > 0 && !f.pinfo) || f.packed_ptr != packed_ptr)
    return set_error(DG_EINVAL, "internal: inconsistent fused write pass");
  hipLaunchKernelGGL(k_fuse_ptr, dim3(1), dim3(64), 0, s, totals_p, f.B, packed_ptr);
  if (f.nblk > 0)
    hipLaunchKernelGGL(k_fuse_write, dim3((unsigned)f.nblk), dim3(MC_THREADS), 0, s, f);
  DG_HIP(hipGetLastError());
  return DG_OK;
}

}  // namespace dg

extern "C" const char *dg_last_error(void) { return dg::g_err; }
extern "C" size_t dg_member_lines_bytes(int64_t num_nodes) {
  return num_nodes < 1 ? 0 : (size_t)dg::mc_touch_bytes(num_nodes);
}
extern "C" const char *dg_version(void) { return "libdg 0.1 (gfx950)"; }
