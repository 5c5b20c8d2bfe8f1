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
