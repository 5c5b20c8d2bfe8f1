// Batched feature packing (DiskGNN §5.2, Fig. 6b) and the interpreted address
// tables (§6), for up to 64 mini-batches at once.
//
// The paper's packer scans the feature table partition by partition in
// consecutive-ID order and appends each needed feature to every mini-batch
// that needs it, so each feature is read once.  Here the table is in HBM and
// the "partition scan" becomes one pass over a node-major membership mask
// (bit b of mask[u] = batch b needs u): that pass yields, in ascending ID
// order, the group's unique set U, the non-cached unique set U_nc, each
// batch's packed order P_b, and for every (u, b) pair of U_nc the packed row
// it goes to.  The gather (dg_gather.hip) then reads each row of U_nc once and
// writes it to all its destination rows.
#include <initializer_list>
#include <mutex>
#include <string.h>

#include "dg_passes.h"
#include "dg_rows.h"

// Scratch of dg_pack_group_noalloc (see scratch_address below).
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)256 << 20;
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

namespace dg {
namespace {

constexpr int THREADS = 256;

struct Lists {
  int B;
  int64_t stride;
  int64_t start[DG_MAX_BATCHES + 1];  // prefix of node counts
};

inline unsigned blocks_for(int64_t n) { return (unsigned)((n + THREADS - 1) / THREADS); }

__global__ __launch_bounds__(THREADS) void k_pack_mark(Lists L, const int32_t *nodes, int64_t N,
                                                       uint64_t *mask, uint32_t *err) {
  int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (i >= L.start[L.B]) return;
  int b = find_batch_wave(L.start, L.B, i);
  int32_t u = nodes[(int64_t)b * L.stride + (i - L.start[b])];
  if (u < 0 || (int64_t)u >= N) {
    atomicOr(err, ERR_NODE_RANGE);
    return;
  }
  // no-return atomic: a node repeated within a batch shows up later as fewer
  // (node, batch) pairs in the mask than list entries
  atomicOr((unsigned long long *)&mask[u], 1ull << b);
}

// packed_ptr from the per-batch totals of the count pass.
__global__ void k_packed_ptr(const int64_t *totals, int B, int64_t *packed_ptr) {
  if (threadIdx.x == 0) {
    int64_t run = 0;
    packed_ptr[0] = 0;
    for (int b = 0; b < B; ++b) {
      run += totals[b];
      packed_ptr[b + 1] = run;
    }
  }
}

// loc_b[j] = -(slot+1) for a cached node, else its rank in P_b.  A non-cached
// node's pairs start at nodeoff[u], one per batch that holds it, in batch
// order, each naming its packed row; the entry takes the first pair whose row
// lies in chunk b and checks that the row is u's (packed_ids).  An entry whose
// node has no such pair (a given membership mask that misses it) is reported,
// so no unchecked address reaches the table.  The mask itself is not read
// here: the count pass may have cleared it already.
// PENDING: loc already holds the sampler's entries; only entries equal to
// DG_LOC_PENDING (non-cached nodes) are completed, and no cache slot is read
// (a pending node that is cached has no pair, and is reported as above).
template <bool PENDING>
__global__ __launch_bounds__(THREADS) void k_build_loc(Lists L, const int32_t *nodes,
                                                       const int32_t *cache_slot,
                                                       const int64_t *nodeoff,
                                                       const int64_t *pairdest, int64_t n_pairs,
                                                       const int32_t *packed_ids,
                                                       const int64_t *packed_ptr, int32_t *loc,
                                                       int64_t N, uint32_t *err) {
  const int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (i >= L.start[L.B]) return;
  const int b = find_batch_wave(L.start, L.B, i);
  const int64_t at = (int64_t)b * L.stride + (i - L.start[b]);
  if (PENDING && loc[at] != (int32_t)DG_LOC_PENDING) return;
  const int32_t u = nodes[at];
  if (u < 0 || (int64_t)u >= N) {
    atomicOr(err, ERR_NODE_RANGE);
    return;
  }
  const int32_t sl = PENDING ? -1 : cache_slot[u];
  int32_t out = 0;
  if (sl >= 0) {
    out = -(sl + 1);
  } else {
    bool found = false;
    int64_t p = nodeoff[u];  // meaningful only for nodes of U_nc; checked below
    if (packed_ids && p >= 0 && p < n_pairs) {
      const int64_t lo = packed_ptr[b], hi = packed_ptr[b + 1];
      const int64_t pend = n_pairs - p > DG_MAX_BATCHES ? p + DG_MAX_BATCHES : n_pairs;
      for (; p < pend; ++p) {
        const int64_t d = pairdest[p];
        if (d < lo) continue;  // a pair of an earlier batch
        if (d < hi && packed_ids[d] == u) {
          out = (int32_t)(d - lo);
          found = true;
        }
        break;
      }
    }
    if (!found) atomicOr(err, ERR_MEMBERSHIP);
  }
  loc[at] = out;
}


}  // namespace

void carve_pack(PackWs &w, Carve &c, int64_t N, int B, int64_t total_nodes) {
  int64_t ucap = total_nodes < N ? total_nodes : N;
  w.err = c.take<uint32_t>(32);
  w.mask = c.take<uint64_t>((size_t)N);
  w.nodeoff = c.take<int64_t>((size_t)N);
  w.unc_ids = c.take<int32_t>((size_t)ucap + 1);
  w.unc_off = c.take<int64_t>((size_t)ucap + 1);
  w.pairdest = c.take<int64_t>((size_t)total_nodes + 1);
  w.ms = MaskScan{};
  w.ms.N = N;
  w.ms.B = B;
  mask_scan_carve(w.ms, c);
}

namespace {

// Device-to-host read of a call's counts: through the library's page-locked
// buffer, or (no_alloc) straight into the host variable.
int read_back(void *dst, const void *src, size_t bytes, hipStream_t s, bool no_alloc) {
  return no_alloc ? read_to_host_unstaged(dst, src, bytes, s) : read_to_host(dst, src, bytes, s);
}

int read_err(uint32_t *err, hipStream_t s, bool no_alloc) {
  uint32_t bits = 0;
  DG_TRY(read_back(&bits, err, sizeof(bits), s, no_alloc));
  if (bits) return set_error(DG_EINVAL, "invalid input data: %s", describe_device_error(bits));
  return DG_OK;
}

}  // namespace

size_t pack_ws_bytes(int64_t num_nodes, int32_t B, int64_t total_nodes) {
  if (num_nodes < 1 || B < 1 || B > DG_MAX_BATCHES || total_nodes < 0) return 0;
  Carve c(nullptr);
  PackWs w;
  carve_pack(w, c, num_nodes, B, total_nodes);
  return c.used;
}

namespace {

// ---------------------------------------------------------------- fixed scratch
// Scratch of dg_pack_group_noalloc: a file-scope device array (one copy per GPU,
// held until the process ends).  Host code never passes the array's name to a
// kernel (on the host it is only a stand-in for the symbol): it asks the runtime
// for the array's device address once per device and uses that.
constexpr int NOALLOC_DEVICES = 16;

int scratch_address(void **out) {
  static std::mutex mu;
  static void *addr[NOALLOC_DEVICES] = {};
  int dev = 0;
  DG_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= NOALLOC_DEVICES)
    return set_error(DG_EHIP, "dg_pack_group_noalloc: device index %d out of range", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(DG_EHIP, "dg_pack_group_noalloc: hipGetSymbolAddress failed: %s",
                       hipGetErrorString(e));
    addr[dev] = p;
  }
  *out = addr[dev];
  return DG_OK;
}

}  // namespace

int pack_impl(const void *feats, int64_t N, int64_t row_bytes, const int32_t *cache_slot,
              int32_t B, const int32_t *nodes, int64_t node_stride, const int64_t *node_count,
              int64_t packed_cap, void *packed, int32_t *packed_ids, int64_t *packed_ptr,
              int64_t *packed_ptr_host, int32_t *loc, int32_t *group_unique, int64_t unique_cap,
              uint64_t *membership, const uint8_t *member_lines, const int32_t *cache_nodes,
              int64_t cache_rows, void *cache_table, uint32_t flags, void *ws,
              size_t ws_bytes, hipStream_t stream, hipStream_t rows_stream, dg_sizes *sizes,
              dg_timing *timing, bool no_alloc) {
  if (!feats || !cache_slot || !nodes || !node_count || !packed_ptr || !packed_ptr_host ||
      !loc || !sizes)
    return set_error(DG_EINVAL, "dg_pack_group: null pointer argument");
  if (cache_table && (!cache_nodes || cache_rows < 0 || !packed ||
                      (flags & DG_PACK_ROWS_STREAM)))
    return set_error(DG_EINVAL, "dg_pack_group: the cache fill needs cache_nodes, "
                                "cache_rows >= 0 and packed, and no DG_PACK_ROWS_STREAM");
  const int64_t n_cache = cache_table ? cache_rows : 0;
  if (N < 1 || N > 0x7fffffffll || row_bytes < 1 || B < 1 || B > DG_MAX_BATCHES ||
      node_stride < 0 || packed_cap < 0 || unique_cap < 0)
    return set_error(DG_EINVAL, "dg_pack_group: bad sizes (N=%lld row_bytes=%lld B=%d)",
                     (long long)N, (long long)row_bytes, B);
  if (flags & ~(DG_PACK_CLEAR_MEMBERSHIP | DG_PACK_ROWS_STREAM | DG_PACK_LOC_PENDING))
    return set_error(DG_EINVAL, "dg_pack_group: unknown flags 0x%x", flags);
  const bool clear_membership = flags & DG_PACK_CLEAR_MEMBERSHIP;
  if (clear_membership && !membership)
    return set_error(DG_EINVAL, "dg_pack_group: DG_PACK_CLEAR_MEMBERSHIP needs membership");
  if (member_lines && !membership)
    return set_error(DG_EINVAL, "dg_pack_group: member_lines needs membership");
  if ((flags & DG_PACK_ROWS_STREAM) && timing)
    return set_error(DG_EINVAL, "dg_pack_group: timing cannot be combined with "
                                "DG_PACK_ROWS_STREAM");
  Lists L;
  L.B = B;
  L.stride = node_stride;
  L.start[0] = 0;
  for (int b = 0; b < B; ++b) {
    if (node_count[b] < 0 || node_count[b] > node_stride)
      return set_error(DG_EINVAL, "dg_pack_group: node_count[%d] = %lld outside [0, %lld]", b,
                       (long long)node_count[b], (long long)node_stride);
    L.start[b + 1] = L.start[b] + node_count[b];
  }
  const int64_t total = L.start[B];
  if (packed_cap > 0 && !packed_ids)
    return set_error(DG_EINVAL, "dg_pack_group: null packed_ids");
  const size_t need_ws = pack_ws_bytes(N, B, total);
  if (no_alloc && need_ws > ws_bytes)
    return set_error(DG_EWORKSPACE,
                     "dg_pack_group_noalloc: these sizes need %zu bytes of scratch, above its "
                     "%zu bytes",
                     need_ws, ws_bytes);
  if (!ws || ws_bytes < need_ws || ((uintptr_t)ws & 255))
    return set_error(DG_EWORKSPACE, "dg_pack_group: workspace needs %zu bytes, 256-aligned",
                     need_ws);

  hipStream_t s = stream;
  PackWs w;
  Carve c(ws);
  carve_pack(w, c, N, B, total);
  w.ms.err = w.err;
  memset(sizes, 0, sizeof(*sizes));
  sizes->max_batch_nodes = sizes->max_batch_edges = sizes->total_edges = -1;
  sizes->total_nodes = total;
  sizes->exact = 1;
  if (timing) memset(timing, 0, sizeof(*timing));
  PhaseTimer tm(timing != nullptr, s);

  int rc;
  const int e0 = tm.mark();
  if ((rc = fill_u64(reinterpret_cast<uint64_t *>(w.err), 16, 0, s))) return rc;
  if (membership) {
    w.mask = membership;  // written only with DG_PACK_CLEAR_MEMBERSHIP
  } else {
    if ((rc = fill_u64(w.mask, (size_t)N, 0, s))) return rc;
    if (total > 0) {
      hipLaunchKernelGGL(k_pack_mark, dim3(blocks_for(total)), dim3(THREADS), 0, s, L, nodes, N,
                         w.mask, w.err);
      DG_HIP(hipGetLastError());
    }
  }
  const int e1 = tm.mark();
  // unique set, packed order, packed_ptr
  int64_t totals[DG_MAX_BATCHES + 5];  // row totals, then the error word
  w.ms.mask = w.mask;
  w.ms.touched = member_lines;  // lines without a member are not read
  w.ms.clear_mask = clear_membership;
  w.ms.cache_slot = cache_slot;
  w.ms.err_stage = w.ms.totals + mc_rows(B);  // staged by the count pass's row scan
  if ((rc = mask_scan_count(w.ms, s))) return rc;
  DG_TRY(read_back(totals, w.ms.totals, sizeof(int64_t) * (mc_rows(B) + 1), s, no_alloc));
  if (totals[mc_rows(B)])
    return set_error(DG_EINVAL, "invalid input data: %s",
                     describe_device_error((uint32_t)totals[mc_rows(B)]));
  int64_t rows = 0;
  packed_ptr_host[0] = 0;
  for (int b = 0; b < B; ++b) {
    rows += totals[b];
    packed_ptr_host[b + 1] = rows;
  }
  sizes->packed_rows = rows;
  sizes->unique_nodes = totals[row_all(B)];
  sizes->unique_packed = totals[row_packed(B)];
  if (rows != totals[row_pairs(B)])
    return set_error(DG_EINVAL, "dg_pack_group: internal pair count mismatch");
  if (totals[row_all_pairs(B)] != total)
    return set_error(DG_EINVAL, "invalid input data: %s",
                     membership ? "the membership mask does not match the node lists (or a node "
                                  "appears twice in one mini-batch)"
                                : describe_device_error(ERR_DUP_NODE));
  if (rows > packed_cap || (group_unique && sizes->unique_nodes > unique_cap))
    return set_error(DG_ECAPACITY,
                     "dg_pack_group: need packed_cap >= %lld and unique_cap >= %lld",
                     (long long)rows, (long long)sizes->unique_nodes);
  hipLaunchKernelGGL(k_packed_ptr, dim3(1), dim3(64), 0, s, w.ms.totals, B, packed_ptr);
  for (int b = 0; b < B; ++b) w.ms.seg_base[b] = packed_ptr_host[b];
  w.ms.seg_out = packed_ids;
  w.ms.uniq_out = group_unique;
  w.ms.unc_ids = w.unc_ids;
  w.ms.unc_off = w.unc_off;
  w.ms.nodeoff = w.nodeoff;
  w.ms.pairdest = w.pairdest;
  if ((rc = mask_scan_write(w.ms, s))) return rc;
  const int e2 = tm.mark();
  // The address tables (random reads) and the fan-out gather (HBM streaming)
  // are independent.  With DG_PACK_ROWS_STREAM the gather goes to the caller's
  // rows_stream and is not waited for.  Otherwise untimed calls run them side by
  // side, the tables on a side stream joined back before the call returns, and
  // timed calls run them one after the other so that each phase has its own
  // time.
  // The row copy also fills the cache table when one is given (the cache as
  // one more mini-batch of the same gather, §5.2).
  const RowCopy rc_rows{feats,      N,      row_bytes,   w.unc_ids, w.unc_off,
                        sizes->unique_packed,  rows, w.pairdest, packed,
                        cache_nodes, n_cache, cache_table, w.err};
  const bool rows_async = (flags & DG_PACK_ROWS_STREAM) && packed;
  SideStream *side = nullptr;
  if (rows_async && total > 0) {
    SideStream *ss = nullptr;
    DG_TRY(side_stream(&ss));
    DG_HIP(hipEventRecord(ss->handoff, s));
    DG_HIP(hipStreamWaitEvent(rows_stream, ss->handoff, 0));
    if ((rc = launch_fanout(rc_rows, rows_stream))) return rc;
  } else if (!timing && !no_alloc && packed && total > 0) {
    DG_TRY(side_stream(&side));
    DG_HIP(hipEventRecord(side->fork, s));
    DG_HIP(hipStreamWaitEvent(side->s, side->fork, 0));
  }
  if (total > 0) {
    const dim3 lg(blocks_for(total)), lb(THREADS);
    hipStream_t ls = side ? side->s : s;
    if (flags & DG_PACK_LOC_PENDING)
      hipLaunchKernelGGL(k_build_loc<true>, lg, lb, 0, ls, L, nodes, cache_slot, w.nodeoff,
                         w.pairdest, rows, packed_ids, packed_ptr, loc, N, w.err);
    else
      hipLaunchKernelGGL(k_build_loc<false>, lg, lb, 0, ls, L, nodes, cache_slot, w.nodeoff,
                         w.pairdest, rows, packed_ids, packed_ptr, loc, N, w.err);
    DG_HIP(hipGetLastError());
  }
  if (side) DG_HIP(hipEventRecord(side->join, side->s));
  const int e3 = tm.mark();
  if (packed && !rows_async &&  // packed == NULL: address tables only, no row copy
      (rc = launch_fanout(rc_rows, s)))
    return rc;
  if (side) DG_HIP(hipStreamWaitEvent(s, side->join, 0));
  const int e4 = tm.mark();
  if ((rc = read_err(w.err, s, no_alloc))) return rc;
  if (timing) {
    timing->mark_ms = tm.ms(e0, e1);
    timing->order_ms = tm.ms(e1, e2);
    timing->loc_ms = tm.ms(e2, e3);
    timing->gather_ms = tm.ms(e3, e4);
    timing->total_ms = tm.ms(e0, e4);
  }
  return DG_OK;
}

namespace {

struct LocFill {
  int B;
  int64_t node_cap;
  int64_t start[DG_MAX_BATCHES + 1];  // packed_ptr
  int64_t n[DG_MAX_BATCHES];          // list lengths
};

// P_b and the address-table entries of the packed pairs after a fused
// compaction: packed row i of chunk b holds node u (low half of pinfo[i]),
// which is entry j of nodes_b, with j the list slot in the high half for a
// pair new at the last hop, else u's local index in the direct table;
// packed_ids[i] = u and loc_b[j] = i - packed_ptr[b], u's rank in P_b.  Every
// non-cached list entry is reached once this way (its pair is in P_b).
__global__ __launch_bounds__(THREADS) void k_loc_packed(LocFill F, const uint64_t *pinfo,
                                                        const int32_t *local,
                                                        int32_t *packed_ids, int32_t *loc,
                                                        uint32_t *err) {
  const int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (i >= F.start[F.B]) return;
  const int b = find_batch_wave(F.start, F.B, i);
  const uint64_t e = pinfo[i];
  const int32_t u = (int32_t)(uint32_t)e;
  int32_t j = (int32_t)(e >> 32);
  packed_ids[i] = u;
  if (j < 0) j = local[(int64_t)u * F.B + b];
  if (j < 0 || (int64_t)j >= F.n[b]) {
    atomicOr(err, ERR_INTERNAL);
    return;
  }
  loc[(int64_t)b * F.node_cap + j] = (int32_t)(i - F.start[b]);
}

}  // namespace

int pack_fused_tail(const FusedTail &t, bool rows_async, hipStream_t s, hipStream_t rows_stream,
                    PhaseTimer *tm, int *ev_loc, int *ev_gather) {
  // The row copy depends only on the write pass's U_nc lists: on a second
  // stream it starts at once, beside the address tables.
  const RowCopy rc_rows{t.feats,   t.N,       t.row_bytes, t.unc_ids, t.unc_off,
                        t.n_unc,   t.rows,    t.pairdest,  t.packed,  nullptr,
                        0,         nullptr,   t.err};
  const bool copy = t.packed && t.n_unc > 0;
  int rc;
  if (copy && rows_async) {
    SideStream *ss = nullptr;
    DG_TRY(side_stream(&ss));
    DG_HIP(hipEventRecord(ss->handoff, s));
    DG_HIP(hipStreamWaitEvent(rows_stream, ss->handoff, 0));
    if ((rc = launch_fanout(rc_rows, rows_stream))) return rc;
  }
  if (t.rows > 0) {
    LocFill F;
    F.B = t.B;
    F.node_cap = t.node_cap;
    for (int b = 0; b <= t.B; ++b) F.start[b] = t.packed_ptr_host[b];
    for (int b = 0; b < t.B; ++b) F.n[b] = t.n_b[b];
    hipLaunchKernelGGL(k_loc_packed, dim3(blocks_for(t.rows)), dim3(THREADS), 0, s, F,
                       t.pinfo, t.local, t.packed_ids, t.loc, t.err);
    DG_HIP(hipGetLastError());
  }
  *ev_loc = tm ? tm->mark() : -1;
  if (copy && !rows_async && (rc = launch_fanout(rc_rows, s))) return rc;
  *ev_gather = tm ? tm->mark() : -1;
  return DG_OK;
}

}  // namespace dg

using namespace dg;

extern "C" size_t dg_pack_workspace_bytes(int64_t num_nodes, int32_t B, int64_t total_nodes) {
  return pack_ws_bytes(num_nodes, B, total_nodes);
}

extern "C" int dg_pack_group(const void *feats, int64_t N, int64_t row_bytes,
                             const int32_t *cache_slot, int32_t B, const int32_t *nodes,
                             int64_t node_stride, const int64_t *node_count, int64_t packed_cap,
                             void *packed, int32_t *packed_ids, int64_t *packed_ptr,
                             int64_t *packed_ptr_host, int32_t *loc, int32_t *group_unique,
                             int64_t unique_cap, uint64_t *membership,
                             const uint8_t *member_lines, const int32_t *cache_nodes,
                             int64_t cache_rows, void *cache_table, uint32_t flags,
                             void *ws, size_t ws_bytes, hipStream_t stream,
                             hipStream_t rows_stream, dg_sizes *sizes, dg_timing *timing) {
  return pack_impl(feats, N, row_bytes, cache_slot, B, nodes, node_stride, node_count,
                   packed_cap, packed, packed_ids, packed_ptr, packed_ptr_host, loc, group_unique,
                   unique_cap, membership, member_lines, cache_nodes, cache_rows, cache_table,
                   flags, ws, ws_bytes, stream, rows_stream, sizes, timing, false);
}

extern "C" size_t dg_pack_noalloc_scratch_bytes(void) { return NOALLOC_SCRATCH_BYTES; }

extern "C" int dg_pack_group_noalloc(const void *feats, int64_t N, int64_t row_bytes,
                                     const int32_t *cache_slot, int32_t B, const int32_t *nodes,
                                     int64_t node_stride, const int64_t *node_count,
                                     int64_t packed_cap, void *packed, int32_t *packed_ids,
                                     int64_t *packed_ptr, int64_t *packed_ptr_host, int32_t *loc,
                                     int32_t *group_unique, int64_t unique_cap,
                                     uint64_t *membership, const uint8_t *member_lines,
                                     const int32_t *cache_nodes, int64_t cache_rows,
                                     void *cache_table, uint32_t flags, hipStream_t stream,
                                     dg_sizes *sizes) {
  if (flags & DG_PACK_ROWS_STREAM)
    return set_error(DG_EINVAL, "dg_pack_group_noalloc: DG_PACK_ROWS_STREAM is not available");
  void *ws = nullptr;
  DG_TRY(scratch_address(&ws));
  return pack_impl(feats, N, row_bytes, cache_slot, B, nodes, node_stride, node_count,
                   packed_cap, packed, packed_ids, packed_ptr, packed_ptr_host, loc, group_unique,
                   unique_cap, membership, member_lines, cache_nodes, cache_rows, cache_table,
                   flags, ws, NOALLOC_SCRATCH_BYTES, stream, nullptr, sizes, nullptr, true);
}
