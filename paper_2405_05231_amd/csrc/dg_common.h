// Internal declarations shared by the libdg translation units (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

#include "dg.h"

namespace dg {

// ---------------------------------------------------------------- errors
// Bits ORed into the device-side error word by data checks.
enum : uint32_t {
  ERR_NODE_RANGE = 1u << 0,  // a seed / node ID outside [0, N)
  ERR_DUP_NODE = 1u << 1,    // a node repeated within one mini-batch
  ERR_CSR = 1u << 2,         // a CSR row with offsets outside [0,E] or decreasing
  ERR_NBR_RANGE = 1u << 3,   // a neighbour ID outside [0, N)
  ERR_CACHE_SLOT = 1u << 4,  // cache_slot[v] < -1
  ERR_ROW_RANGE = 1u << 5,   // an address-table entry outside its table
  ERR_INTERNAL = 1u << 6,    // an internal table overflowed (a library bug)
  ERR_MEMBERSHIP = 1u << 7,  // a given membership mask misses a list entry
};

int set_error(int status, const char *fmt, ...);
const char *describe_device_error(uint32_t bits);

#define DG_HIP(call)                                                              \
  do {                                                                            \
    hipError_t e_ = (call);                                                       \
    if (e_ != hipSuccess)                                                         \
      return ::dg::set_error(DG_EHIP, "%s failed: %s", #call, hipGetErrorString(e_)); \
  } while (0)

#define DG_TRY(call)                  \
  do {                                \
    const int r_ = (call);            \
    if (r_ != DG_OK) return r_;       \
  } while (0)

// ---------------------------------------------------------------- workspace
// Bump allocator over the caller's workspace (256-byte aligned pieces).
struct Carve {
  char *base;
  size_t used = 0;
  explicit Carve(void *p) : base(static_cast<char *>(p)) {}
  template <typename T>
  T *take(size_t count) {
    T *p = reinterpret_cast<T *>(base ? base + used : nullptr);
    used += (count * sizeof(T) + 255) & ~size_t(255);
    return p;
  }
};

// ---------------------------------------------------------------- wave64 helpers
__device__ __forceinline__ int lane_id() { return __lane_id(); }
__device__ __forceinline__ uint64_t lanes_below() { return (1ull << lane_id()) - 1ull; }

template <typename T>
__device__ __forceinline__ T wave_incl_sum(T x) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    T y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

// Wave-wide OR / inclusive sum through the device library's DPP reductions
// (no LDS round trip).
extern "C" __device__ uint64_t __ockl_wfred_or_u64(uint64_t);
extern "C" __device__ int32_t __ockl_wfscan_add_i32(int32_t, bool inclusive);
extern "C" __device__ int32_t __ockl_wfred_add_i32(int32_t);

__device__ __forceinline__ uint64_t wave_or(uint64_t x) { return __ockl_wfred_or_u64(x); }
__device__ __forceinline__ int32_t wave_incl_sum_i32(int32_t x) {
  return __ockl_wfscan_add_i32(x, true);
}

// Value of x in lane `src`, where src is the same in every lane (v_readlane).
__device__ __forceinline__ int64_t read_lane(int64_t x, int src) {
  uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, src);
  uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)x >> 32), src);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Binary search over a non-decreasing prefix array p[0..n] (p[0] = 0): the
// batch b with p[b] <= i < p[b+1].
__device__ __forceinline__ int find_batch(const int64_t *p, int n, int64_t i) {
  int lo = 0, hi = n;  // invariant p[lo] <= i < p[hi]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (p[mid] <= i) lo = mid; else hi = mid;
  }
  return lo;
}

// The same for a wave whose active lanes hold non-decreasing i (lane order):
// when its first and last active lanes fall in one batch, which is the case
// for all but the waves at batch boundaries, the search runs once on values
// that are the same across the wave (scalar loads, no per-lane chain of
// dependent loads); otherwise every lane searches.
__device__ __forceinline__ int find_batch_wave(const int64_t *p, int n, int64_t i) {
  const uint64_t act = __ballot(1);
  const int first = __builtin_ctzll(act), last = 63 - __builtin_clzll(act);
  const int64_t lo = read_lane(i, first), hi = read_lane(i, last);
  int b = 0, top = n;  // invariant p[b] <= lo < p[top]
  while (top - b > 1) {
    const int mid = (b + top) >> 1;
    if (p[mid] <= lo) b = mid; else top = mid;
  }
  if (hi < p[b + 1]) return b;
  return find_batch(p, n, i);
}

// ---------------------------------------------------------------- XCD-aware block order
// The hardware hands consecutive blocks of a grid to the 8 XCDs (each with its
// own L2) in turn.  xcd_block(i, n) renumbers block i so that each XCD takes one
// contiguous run of the n block numbers (a bijection on [0, n) for any n): work
// whose outputs are laid out in block order then writes neighbouring lines from
// one L2, where partial lines merge before they reach HBM.
constexpr int NUM_XCD = 8;
__device__ __forceinline__ uint32_t xcd_block(uint32_t i, uint32_t n) {
  const uint32_t x = i % NUM_XCD, k = i / NUM_XCD;
  const uint32_t q = n / NUM_XCD, r = n % NUM_XCD;
  return x * q + (x < r ? x : r) + k;
}

// ---------------------------------------------------------------- local-index table
// (node u, batch b) -> local index j of u in batch b's node list.  Open
// addressing with linear probing over 2^bits 64-bit slots; an entry is
// key << LT_VALUE_BITS | j with key = u*64 + b + 1 (never 0, so 0 = empty).
// Sized for a load factor of at most 1/2, so probes end quickly.
constexpr int LT_VALUE_BITS = 27;
constexpr int64_t LT_MAX_VALUE = (1ll << LT_VALUE_BITS) - 1;

struct LocalTable {
  uint64_t *slots;
  int bits;
};

__host__ __device__ inline uint64_t lt_key(int32_t u, int b) {
  return (((uint64_t)(uint32_t)u << 6) | (uint64_t)b) + 1ull;
}
__device__ __forceinline__ uint64_t lt_slot(const LocalTable &t, uint64_t key) {
  return (key * 0x9E3779B97F4A7C15ull) >> (64 - t.bits);  // Fibonacci hashing
}
// Returns false only if the table is full (cannot happen at the sizes used).
__device__ __forceinline__ bool lt_insert(const LocalTable &t, int32_t u, int b, int64_t j) {
  const uint64_t key = lt_key(u, b);
  const uint64_t e = (key << LT_VALUE_BITS) | (uint64_t)j;
  const uint64_t m = (1ull << t.bits) - 1ull;
  uint64_t s = lt_slot(t, key);
  for (uint64_t probe = 0; probe <= m; ++probe, s = (s + 1) & m) {
    unsigned long long old =
        atomicCAS((unsigned long long *)&t.slots[s], 0ull, (unsigned long long)e);
    if (old == 0ull) return true;
  }
  return false;
}
// Local index of (u, b), or -1 if absent.
__device__ __forceinline__ int64_t lt_find(const LocalTable &t, int32_t u, int b) {
  const uint64_t key = lt_key(u, b);
  const uint64_t m = (1ull << t.bits) - 1ull;
  uint64_t s = lt_slot(t, key);
  for (uint64_t probe = 0; probe <= m; ++probe, s = (s + 1) & m) {
    const uint64_t e = t.slots[s];
    if (e == 0ull) return -1;
    if ((e >> LT_VALUE_BITS) == key) return (int64_t)(e & (uint64_t)LT_MAX_VALUE);
  }
  return -1;
}
inline int lt_bits_for(int64_t entries) {
  int bits = 10;
  while ((1ll << bits) < 2 * entries) ++bits;
  return bits;
}

// ---------------------------------------------------------------- host reads
// Copies `bytes` from device memory to host memory after the stream's earlier
// work and waits for it.  Small reads go through a page-locked buffer kept per
// host thread (allocated on first use, held until the process ends), which
// shortens each round trip; otherwise the copy goes to dst directly.
int read_to_host(void *dst, const void *src, size_t bytes, hipStream_t s);
// The same straight into dst (pageable or not), with no buffer of the library's.
int read_to_host_unstaged(void *dst, const void *src, size_t bytes, hipStream_t s);

// ---------------------------------------------------------------- side stream
// A second stream per host thread and device, for kernels a call runs beside
// the caller's stream, with the events that fork from and join back to it (and
// one that orders work the caller's second stream runs behind the call's).
// Created on first use at default priority and held until the process ends.
struct SideStream {
  hipStream_t s;
  hipEvent_t fork, join, handoff;
};
int side_stream(SideStream **out);

// ---------------------------------------------------------------- fill / scan
int fill_u64(uint64_t *p, size_t n, uint64_t value, hipStream_t s);

// Exclusive scan of n int64 values: out[0..n] (out[n] = total).  tile_sums needs
// scan_tile_count(n) entries.
size_t scan_tile_count(int64_t n);
int scan_exclusive(const int64_t *in, int64_t *out, int64_t n, int64_t *tile_sums,
                   hipStream_t s);

// ---------------------------------------------------------------- mask compaction
// A node-major membership mask: bit b of mask[u] says that node u belongs to
// mini-batch b.  A block of MC_WAVES waves owns MC_BLOCK_NODES consecutive
// nodes; wave w owns the w-th run of MC_TILE of them, and round r of a wave
// covers nodes tile0 + r*64 + lane, so (wave, round, lane) order is node order.
constexpr int MC_WAVES = 4;
constexpr int MC_THREADS = 64 * MC_WAVES;
constexpr int MC_ROUNDS = 16;
constexpr int MC_TILE = 64 * MC_ROUNDS;
constexpr int MC_BLOCK_NODES = MC_TILE * MC_WAVES;
constexpr int MC_CHUNK = 64;  // blocks per chunk of the row scan
// Touched marks: one byte per 2^MC_TOUCH_SHIFT consecutive nodes (one 64-byte
// line of the mask).
constexpr int MC_TOUCH_SHIFT = 3;

__host__ __device__ inline int64_t mc_blocks(int64_t N) { return (N + MC_BLOCK_NODES - 1) / MC_BLOCK_NODES; }
__host__ __device__ inline int64_t mc_chunks(int64_t nblk) { return (nblk + MC_CHUNK - 1) / MC_CHUNK; }
__host__ __device__ inline int64_t mc_touch_bytes(int64_t N) {
  return mc_blocks(N) * (MC_BLOCK_NODES >> MC_TOUCH_SHIFT);
}

// Count-matrix rows: [0,B) per batch (non-cached members), then:
__host__ __device__ inline int row_all(int B) { return B; }        // nodes with any bit set (U)
__host__ __device__ inline int row_packed(int B) { return B + 1; } // ... and not cached (U_nc)
__host__ __device__ inline int row_pairs(int B) { return B + 2; }  // (node, batch) pairs of U_nc nodes
__host__ __device__ inline int row_all_pairs(int B) { return B + 3; }  // all (node, batch) pairs
__host__ __device__ inline int mc_rows(int B) { return B + 4; }

struct MaskScan {
  uint64_t *mask;
  const int32_t *cache_slot;  // nullable: no node is cached
  int64_t N;
  int B;
  int64_t nblk;        // blocks of MC_BLOCK_NODES nodes
  uint32_t *cnt;       // [nblk][rows] per-block counts
  uint32_t *wpre;      // [nblk][MC_WAVES][rows] each wave's exclusive prefix in its block
  uint32_t *wcnt;      // [nblk][MC_WAVES] non-empty words of each wave's tile
  uint64_t *cw_mask;   // [nblk][MC_WAVES][MC_TILE] those words (count pass -> write pass)
  uint16_t *cw_off;    // ... their node offsets in the tile; bit 15 = cached
  int64_t *base;       // [nblk][rows] exclusive scans down each row
  int64_t *chunk_sum;  // [chunks][rows]
  int64_t *totals;     // [rows]
  uint32_t *err;
  int64_t *err_stage;  // nullable: receives *err after the count pass (for the read-back)
  // write pass outputs (which are required depends on the mode, see below)
  int64_t seg_base[DG_MAX_BATCHES];  // start index of batch b's list in seg_out
  int64_t seg_end[DG_MAX_BATCHES];   // sampling: end of batch b's room in seg_out
  int32_t *seg_out;                  // per-batch ascending lists of non-cached members
  int32_t *uniq_out;                 // U ascending
  int32_t *unc_ids;                  // U_nc ascending
  int64_t *unc_off;                  // first pair of each U_nc node
  int64_t *nodeoff;                  // [N] first pair of node u (U_nc nodes only)
  int64_t *pairdest;                 // per pair: seg_base[b] + rank of u in b's list
  int32_t *local_out;                // [N][B]: local index of (u, b) = local_base[b] + rank
  int64_t local_base[DG_MAX_BATCHES];
  uint64_t *prev;                    // nullable: members already listed; the passes
                                     // see mask & ~prev, and the count pass adds
                                     // the new bits to prev
  bool keep_prev;                    // false: leave prev as it is (nothing reads it later)
  bool clear_prev;                   // (without keep_prev) zero each non-zero prev word read
  bool clear_mask;                   // zero each non-zero mask word read (packing mode)
  uint8_t *lines_out;                // sampling, whole sweeps only (nullable): a byte per
                                     // 2^MC_TOUCH_SHIFT nodes, non-zero iff one of them
                                     // holds a bit of the (keep-masked) mask
  const uint8_t *touched;            // nullable: a byte per 2^MC_TOUCH_SHIFT nodes
                                     // (mc_touch_bytes(N) in all); nodes whose byte
                                     // is 0 hold no bit to list (not read)
  // sampling only (both or neither): for each listed pair, the address-table
  // entry at the same index as its seg_out slot: -(loc_slot[u]+1) for a cached
  // node, DG_LOC_PENDING otherwise
  const int32_t *loc_slot;
  int32_t *loc_out;
  // The write pass runs in one of two modes: packing (pairdest set: seg_out,
  // unc_ids, unc_off, nodeoff required, uniq_out optional, cached nodes left out
  // of the lists) or sampling (pairdest NULL: prev and seg_out required,
  // local_out and loc_slot/loc_out optional, no cache_slot).
};


size_t mask_scan_ws_bytes(int64_t N, int B);
void mask_scan_carve(MaskScan &m, Carve &c);
// Count pass + per-row scans (asynchronous); m.totals[row] receives each row's
// total (B+4 values) on the device.
int mask_scan_count(MaskScan &m, hipStream_t s);
// Write pass (uses the scans of the preceding count pass).
int mask_scan_write(const MaskScan &m, hipStream_t s);
// Member lines of the whole mask (mc_touch_bytes(N) bytes), by a pass of its own.
int member_lines_pass(const uint64_t *mask, int64_t N, int B, uint8_t *out, hipStream_t s);
// The row scans of a count matrix filled by a count pass (part of mask_scan_count).
int mask_scan_rows(MaskScan &m, hipStream_t s);

// ---------------------------------------------------------------- fused compaction
// The last sampling hop's count and write passes doing batched packing's pass
// over the membership words as well (dg_sample_pack_group).  The mask then
// holds every (node, batch) pair of the group and prev the pairs listed before
// the last hop, so one sweep gives both the hop's new pairs (m & ~prev) and
// packing's sets.  The compact list holds every non-empty word: m, its new
// bits and its offset (bit 15 = cached).  Two count matrices come out of the
// count pass, each scanned by the row scans of a MaskScan view of its own:
//   s: rows [0, B) = new pairs per batch (the other four rows as in sampling);
//   p: packing's rows ([0, B) non-cached pairs per batch, U, U_nc, non-cached
//      pairs, all pairs).
// The count pass zeroes every mask word it reads, and the prev words too with
// clear_prev.  The write pass writes sampling's lists and the address-table
// entries of new cached pairs, and packing's U, U_nc, pair offsets and pair
// destinations; for every packed pair it records the node and, when the pair
// is new at this hop, its list slot (pinfo), from which the address tables
// and P_b follow.  Every index is checked against its buffer:
// counts beyond a capacity are found by the host after the read-back.
struct FuseScan {
  uint64_t *mask;
  uint64_t *prev;
  const int32_t *cache_slot;
  int64_t N;
  int B;
  int64_t nblk;
  bool clear_prev;
  uint32_t *err;
  // compact list (the sampling view's arrays, and the packing view's cw_mask
  // for the new bits)
  uint32_t *wcnt;
  uint64_t *cw_mask;
  uint64_t *cw_new;
  uint16_t *cw_off;
  int32_t *cw_slot;  // cache slot of each listed word's node (-1: not cached)
  uint32_t *cnt_s, *wpre_s, *cnt_p, *wpre_p;
  const int64_t *base_s, *base_p;
  // write pass, sampling: the hop's segments of the node lists
  int64_t node_cap;
  int64_t seg_base[DG_MAX_BATCHES];  // b*node_cap + n_b before the hop
  int64_t seg_end[DG_MAX_BATCHES];   // (b+1)*node_cap
  int32_t *seg_out;
  int32_t *loc_out;    // [B*node_cap] address tables (cached entries written here)
  int32_t *local_out;  // nullable: [N][B] local indices of the hop's pairs
  // write pass, packing
  const int64_t *packed_ptr;  // device [B+1], from the p view's totals
  int64_t packed_cap;         // entries of pinfo
  uint64_t *pinfo;            // per packed row: node ID (low half) and the pair's
                              // list slot if new at this hop, else -1 (high half)
  int32_t *uniq_out;  // nullable
  int64_t unique_cap;
  int32_t *unc_ids;
  int64_t *unc_off;
  int64_t unc_cap;
  int64_t *nodeoff;  // nullable
  int64_t *pairdest;
  int64_t pair_cap;
};
// Count pass + the row scans of both views (asynchronous).
int fuse_scan_count(const FuseScan &f, MaskScan &vs, MaskScan &vp, hipStream_t s);
// Write pass (after the count pass): first packed_ptr (= f.packed_ptr, B+1
// entries) from the p view's per-batch totals, then the pass itself.
int fuse_scan_write(const FuseScan &f, const int64_t *totals_p, int64_t *packed_ptr,
                    hipStream_t s);

// ---------------------------------------------------------------- packing state
// Workspace of batched packing (also carved by dg_sample_pack_group).
struct PackWs {
  uint32_t *err;
  uint64_t *mask;
  int64_t *nodeoff;
  int32_t *unc_ids;
  int64_t *unc_off;
  int64_t *pairdest;
  MaskScan ms;
};
void carve_pack(PackWs &w, Carve &c, int64_t N, int B, int64_t total_nodes);
size_t pack_ws_bytes(int64_t num_nodes, int32_t B, int64_t total_nodes);
// dg_pack_group's body (no_alloc: dg_pack_group_noalloc's rules).
int pack_impl(const void *feats, int64_t N, int64_t row_bytes, const int32_t *cache_slot,
              int32_t B, const int32_t *nodes, int64_t node_stride, const int64_t *node_count,
              int64_t packed_cap, void *packed, int32_t *packed_ids, int64_t *packed_ptr,
              int64_t *packed_ptr_host, int32_t *loc, int32_t *group_unique, int64_t unique_cap,
              uint64_t *membership, const uint8_t *member_lines, const int32_t *cache_nodes,
              int64_t cache_rows, void *cache_table, uint32_t flags, void *ws,
              size_t ws_bytes, hipStream_t stream, hipStream_t rows_stream, dg_sizes *sizes,
              dg_timing *timing, bool no_alloc);
// What follows a fused compaction: P_b (packed_ids) and the address-table
// entries of the packed pairs, loc[b*node_cap + j] = r for packed row
// packed_ptr[b] + r, with j the list slot in the row's pinfo for a pair new at
// the last hop, else local[u*B + b]; then the row copy (on rows_stream, not
// waited for, when rows_async).
struct PhaseTimer;
struct FusedTail {
  const void *feats;
  int64_t N, row_bytes;
  int B;
  int64_t node_cap;
  const int64_t *n_b;              // [host] list lengths
  const int64_t *packed_ptr_host;  // [host] B+1
  const uint64_t *pinfo;
  const int32_t *local;
  int32_t *packed_ids;
  int32_t *loc;
  void *packed;  // nullable: no row copy
  const int32_t *unc_ids;
  const int64_t *unc_off, *pairdest;
  int64_t n_unc, rows;
  uint32_t *err;
};
int pack_fused_tail(const FusedTail &t, bool rows_async, hipStream_t s, hipStream_t rows_stream,
                    PhaseTimer *tm, int *ev_loc, int *ev_gather);

// ---------------------------------------------------------------- timing
// Events are taken from a pool per host thread and device, created on first
// use and reused by later calls (creating events inside a timed call would
// delay its launches).  A call reads its times only after its final
// synchronisation, and calls on one thread do not overlap, so reuse is safe.
constexpr int TIMER_EVENTS = 24;
constexpr int TIMER_DEVICES = 16;
struct EventPool {
  hipEvent_t ev[TIMER_EVENTS];
  int made = 0;
};
inline EventPool *event_pool() {
  static thread_local EventPool p[TIMER_DEVICES];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= TIMER_DEVICES) return nullptr;
  return &p[dev];
}

struct PhaseTimer {
  bool on;
  hipStream_t s;
  EventPool *p = nullptr;
  int used = 0;
  explicit PhaseTimer(bool enable, hipStream_t st) : on(enable), s(st) {
    if (on) p = event_pool();
    if (!p) on = false;
  }
  int mark() {  // returns the index of a new recorded event, or -1
    if (!on || used >= TIMER_EVENTS) return -1;
    if (used >= p->made) {
      if (hipEventCreate(&p->ev[p->made]) != hipSuccess) return -1;
      ++p->made;
    }
    if (hipEventRecord(p->ev[used], s) != hipSuccess) return -1;
    return used++;
  }
  float ms(int a, int b) const {
    if (!on || a < 0 || b < 0) return 0.f;
    float t = 0.f;
    (void)hipEventElapsedTime(&t, p->ev[a], p->ev[b]);
    return t;
  }
};

}  // namespace dg
