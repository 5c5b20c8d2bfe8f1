// Internal interfaces of the membership-mask passes (sampling's per-hop
// compaction, packing's group pass and the two fused at the last hop) and of
// packing's host side, shared by the library's sources.
#pragma once

#include "dg_common.h"

namespace dg {

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
  uint8_t *plines;                   // nullable (with prev): a byte per 2^MC_TOUCH_SHIFT
                                     // nodes, non-zero iff one of them holds a prev bit;
                                     // prev is read only in marked lines.  With keep_prev
                                     // the pass marks the lines of the new words, with
                                     // clear_prev it zeroes the marks of its tiles
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
  uint8_t *plines;  // nullable: prev's lines, as MaskScan::plines (zeroed with clear_prev)
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

}  // namespace dg
