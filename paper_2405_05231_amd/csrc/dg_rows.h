// Feature-row movement shared by the packing gather and the assembly kernel.
//
// A feature row is row_bytes opaque bytes.  When row_bytes and every base
// pointer are multiples of 16 the row moves as C = row_bytes/16 uint4 vectors;
// a group of LPR lanes owns one row and each lane moves CPL vectors of it
// (vector c of the row goes to lane c % LPR), so each load instruction of a
// group covers LPR*16 contiguous bytes.  Each group handles UNROLL rows per
// iteration and issues all their loads before any store, to keep enough bytes
// in flight to cover HBM latency.  Other sizes take a narrower word and one
// wave per row.
#pragma once

#include "dg_common.h"

namespace dg {

struct RowShape {
  int lpr;  // lanes per row
  int cpl;  // vectors per lane
};

// Launch shapes of the 16-byte path, by vectors per row (C).
inline bool row_shape16(int64_t C, RowShape *s) {
  if (C <= 4) { *s = {4, 1}; return true; }
  if (C <= 8) { *s = {8, 1}; return true; }
  if (C <= 16) { *s = {16, 1}; return true; }
  if (C <= 32) { *s = {32, 1}; return true; }
  if (C <= 64) { *s = {64, 1}; return true; }
  if (C <= 128) { *s = {64, 2}; return true; }
  if (C <= 256) { *s = {64, 4}; return true; }
  return false;  // longer rows: generic path
}

// Rows in flight per lane group: four for rows of one vector per lane, two
// when each lane moves two or more vectors of a row (keeps registers, and so
// occupancy, in check for wide rows).
__host__ __device__ constexpr int rows_in_flight(int cpl) { return cpl >= 2 ? 2 : 4; }

inline int word_bytes(int64_t row_bytes, std::initializer_list<const void *> ptrs) {
  int w = 16;
  auto fits = [&](int a) {
    if (row_bytes % a) return false;
    for (const void *p : ptrs)
      if (p && ((uintptr_t)p % a)) return false;
    return true;
  };
  while (w > 1 && !fits(w)) w >>= 1;
  return w;
}

// 16-byte row vector as a native vector type, so the nontemporal builtins
// apply: every row is read once and written once, so neither side should
// displace reusable lines from the caches.
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4u ld_stream(const v4u *p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_stream(v4u x, v4u *p) { __builtin_nontemporal_store(x, p); }

// The row copy of one packing call: the fan-out gather over U_nc, plus the
// cache rows when a cache table is given.
struct RowCopy {
  const void *X;
  int64_t N, row_bytes;
  const int32_t *ids;
  const int64_t *off;
  int64_t n, pairs;
  const int64_t *dest;
  void *packed;
  const int32_t *cache_nodes;
  int64_t n_cache;
  void *cache_table;
  uint32_t *err;
};
// Launches the fan-out gather of one RowCopy on stream s (nothing when it has
// no item); DG_EHIP when the launch fails.
int launch_fanout(const RowCopy &r, hipStream_t s);

template <typename T>
__device__ __forceinline__ T zero_word() {
  T z;
  memset(&z, 0, sizeof(T));
  return z;
}

}  // namespace dg
