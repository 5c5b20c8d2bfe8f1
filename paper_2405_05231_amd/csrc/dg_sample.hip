// Group sampling: node-wise fan-out neighbour sampling (DiskGNN §2, Fig. 1) for
// up to 64 mini-batches in one pass (offline sampling, §3).
//
// Device state: a node-major membership mask visited[u] (bit b = u is in
// mini-batch b) and its copy prev[u] as of the start of the current hop.  A
// hop is:
//   degree pass over the frontier -> exclusive scan (edge slots) ->
//   draw + mark: 1-8 lanes per frontier node, a fire-and-forget atomicOr on
//     visited per sampled edge; a hop that can reach only a small share of the
//     nodes also marks the 8-node lines of the mask it touches ->
//   compaction of visited & ~prev (the nodes new at this hop) into each
//     batch's new segment, ascending, with no sort; it also brings prev up to
//     date (the last hop instead clears prev with DG_SAMPLE_EXIT_CLEAR, and
//     writes the member-lines map when asked) ->
//   one read-back of the hop's counts.
// Sampled neighbours are relabelled from global to local IDs at the end,
// through one of two tables: a direct [N][B] array of local indices that the
// compaction fills as it assigns them (DG_SAMPLE_DIRECT), or a (node, batch)
// hash table sized for the group and filled after the last hop.
#include <string.h>

#include <type_traits>

#include "dg_passes.h"

namespace dg {
namespace {

constexpr int THREADS = 256;
constexpr int FMAX = 32;  // fan-outs up to this take the register path

__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
constexpr uint64_t GAMMA = 0x9E3779B97F4A7C15ull;

// Per-hop description of the frontier, passed by value.
struct Hop {
  int B;
  int32_t f;        // fan-out of this hop (< 0: all)
  int32_t k;        // hop number, 1-based (RNG key)
  int64_t ftot;     // frontier entries over all batches
  int64_t fstart[DG_MAX_BATCHES + 1];  // prefix of frontier sizes
  int64_t fpos[DG_MAX_BATCHES];        // local position of b's first frontier node
  int64_t ebase[DG_MAX_BATCHES];       // edges of b before this hop
  uint64_t bstate[DG_MAX_BATCHES];     // mix64(rng_seed + gamma*(g+1)) per batch
  uint8_t *touched;                    // nullable: a byte per 2^MC_TOUCH_SHIFT nodes, set
                                       // for every node that gains a membership bit
};

// Flattened (batch, position) ranges, for passes over all edge lists, with
// each batch's node count.
struct Lists {
  int B;
  int64_t start[DG_MAX_BATCHES + 1];
  int64_t n[DG_MAX_BATCHES];
};

// Seeds -> node lists, membership bits and local indices; with loc, also the
// seeds' address-table entries (final for cached seeds, pending otherwise).
__global__ __launch_bounds__(THREADS) void k_seed_init(const int32_t *seeds, int B, int S,
                                                       int64_t N, int64_t node_cap,
                                                       int32_t *nodes, uint64_t *visited,
                                                       uint64_t *prev, uint8_t *plines,
                                                       int32_t *local, const int32_t *cache_slot,
                                                       int32_t *loc, uint32_t *err) {
  int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (i >= (int64_t)B * S) return;
  int b = (int)(i / S);
  int64_t j = i - (int64_t)b * S;
  int32_t v = seeds[i];
  nodes[(int64_t)b * node_cap + j] = v;
  if (v < 0 || (int64_t)v >= N) {
    atomicOr(err, ERR_NODE_RANGE);
    return;
  }
  if (loc) {
    const int32_t sl = cache_slot[v];
    if (sl < -1) atomicOr(err, ERR_CACHE_SLOT);
    loc[(int64_t)b * node_cap + j] = sl >= 0 ? -(sl + 1) : (int32_t)DG_LOC_PENDING;
  }
  unsigned long long bit = 1ull << b;
  unsigned long long old = atomicOr((unsigned long long *)&visited[v], bit);
  if (old & bit) atomicOr(err, ERR_DUP_NODE);
  atomicOr((unsigned long long *)&prev[v], bit);  // seeds are not new at hop 1
  plines[v >> MC_TOUCH_SHIFT] = 1;
  if (local) local[(int64_t)v * B + b] = (int32_t)j;
}

__global__ __launch_bounds__(THREADS) void k_frontier_degree(
    Hop h, const int32_t *nodes, int64_t node_cap, const int64_t *off, int64_t N, int64_t E,
    int64_t *f_off, int64_t *f_deg, int64_t *f_cnt, uint32_t *err) {
  int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (i >= h.ftot) return;
  int b = find_batch_wave(h.fstart, h.B, i);
  int32_t v = nodes[(int64_t)b * node_cap + h.fpos[b] + (i - h.fstart[b])];
  int64_t o0 = 0, d = 0;
  if (v >= 0 && (int64_t)v < N) {
    o0 = off[v];
    int64_t o1 = off[v + 1];
    if (o0 < 0 || o1 < o0 || o1 > E) {
      atomicOr(err, ERR_CSR);
    } else {
      d = o1 - o0;
    }
  }
  f_off[i] = o0;
  f_deg[i] = d;
  f_cnt[i] = (h.f < 0 || d <= (int64_t)h.f) ? d : (int64_t)h.f;
}

// Emits up to EMIT sampled edges whose neighbour IDs are already loaded: the
// edge stores, then a fire-and-forget atomicOr of the batch's bit into each
// neighbour's membership word (setting a bit that is already set changes
// nothing, and skipping the atomic for seen pairs would cost a dependent read
// of the word, which measures slower than the atomics it saves).
constexpr int EMIT = 8;

__device__ __forceinline__ void emit_chunk(const int32_t (&u)[EMIT], const int64_t (&slot)[EMIT],
                                           int cnt, int b, int32_t parent, int32_t *edge_src,
                                           int32_t *edge_dst, uint64_t *visited, int64_t N,
                                           uint8_t *touched, uint32_t *err) {
  const unsigned long long bit = 1ull << b;
#pragma unroll
  for (int k = 0; k < EMIT; ++k) {
    if (k < cnt) {
      edge_src[slot[k]] = parent;
      edge_dst[slot[k]] = u[k];
    }
  }
#pragma unroll
  for (int k = 0; k < EMIT; ++k) {
    if (k >= cnt) continue;
    if (u[k] >= 0 && (int64_t)u[k] < N) {
      atomicOr((unsigned long long *)&visited[u[k]], bit);
      if (touched) touched[u[k] >> MC_TOUCH_SHIFT] = 1;
    } else {
      atomicOr(err, ERR_NBR_RANGE);
    }
  }
}

// LPN lanes per frontier node (LPN = 1, 2, 4 or 8; more lanes when the
// frontier is small, so that short hops still keep enough loads in flight).
// Floyd's subset is built in registers (fully unrolled, so the arrays stay in
// VGPRs) when f <= FM, by every lane of the node; FM (8, 16 or 32) is the
// smallest capacity that holds the hop's fan-out, since the arrays' registers
// bound the waves per SIMD and so the loads in flight; each drawn position's rank among the f
// positions gives its slot, so no sort is needed, and lane `sub` takes the
// draws s with s mod LPN = sub.  Neighbour loads and membership atomics are
// issued EMIT at a time so their latencies overlap.  estart[b] = f_eoff at
// batch b's first frontier entry (written on the device by k_batch_bounds).  A
// node whose edges would pass edge_cap writes nothing; the host sees the
// overflow in the edge counts and reports it.
template <int LPN, int FM>
__global__ __launch_bounds__(THREADS) void k_hop_sample(
    Hop h, const int32_t *nodes, int64_t node_cap, const int32_t *idx, const int64_t *f_off,
    const int64_t *f_deg, const int64_t *f_eoff, const int64_t *estart, int64_t edge_cap,
    int32_t *edge_src, int32_t *edge_dst, uint64_t *visited, int64_t N, uint32_t *err) {
  const int64_t t = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  const int64_t i = t / LPN;
  const int sub = (int)(t % LPN);
  if (i >= h.ftot) return;
  int b = find_batch_wave(h.fstart, h.B, i);
  int64_t p = h.fpos[b] + (i - h.fstart[b]);
  int64_t o0 = f_off[i], d = f_deg[i];
  const int64_t first = h.ebase[b] + (f_eoff[i] - estart[b]);  // local index of the 1st edge
  const int64_t cnt = (h.f < 0 || d <= (int64_t)h.f) ? d : (int64_t)h.f;
  if (first + cnt > edge_cap) return;
  int64_t base = (int64_t)b * edge_cap + first;
  int32_t parent = (int32_t)p;
  int32_t u[EMIT];
  int64_t slot[EMIT];
  if (h.f < 0 || d <= (int64_t)h.f) {  // every neighbour, in CSR order
    // lane sub takes positions q0 + sub + LPN*k, so the lanes of a node read
    // consecutive positions in one instruction
    for (int64_t q0 = 0; q0 < d; q0 += (int64_t)LPN * EMIT) {
      int n = 0;
#pragma unroll
      for (int k = 0; k < EMIT; ++k) {
        const int64_t q = q0 + sub + (int64_t)LPN * k;
        slot[k] = base + q;
        u[k] = q < d ? idx[o0 + q] : 0;
        n += q < d ? 1 : 0;
      }
      emit_chunk(u, slot, n, b, parent, edge_src, edge_dst, visited, N, h.touched, err);
    }
    return;
  }
  const int32_t f = h.f;
  int32_t v = nodes[(int64_t)b * node_cap + p];
  uint64_t key = mix64(h.bstate[b] ^ (((uint64_t)(uint32_t)h.k << 32) | (uint64_t)(uint32_t)v));
  if (d > 0x7fffffffll) {  // positions are kept as 32-bit values
    if (sub == 0) atomicOr(err, ERR_CSR);
    return;
  }
  if (f <= FM) {
    uint32_t r[FM];
#pragma unroll
    for (int s = 0; s < FM; ++s) {
      r[s] = 0xffffffffu;
      if (s < f) {
        uint32_t j = (uint32_t)(d - f + s);
        uint64_t hs = mix64(key + GAMMA * (uint64_t)(s + 1));
        uint32_t tt = (uint32_t)__umul64hi(hs, (uint64_t)j + 1ull);
        bool seen = false;
#pragma unroll
        for (int m = 0; m < s; ++m) seen |= (r[m] == tt);
        r[s] = seen ? j : tt;
      }
    }
    // this lane's draws: s = j*LPN + sub for j = 0, 1, ... (a static j, so the
    // register arrays are indexed by constants only)
    constexpr int SPL = FM / LPN;
    uint32_t rv[SPL];
#pragma unroll
    for (int j = 0; j < SPL; ++j) {
      rv[j] = 0xffffffffu;
#pragma unroll
      for (int q = 0; q < LPN; ++q)
        if (q == sub) rv[j] = r[j * LPN + q];
    }
#pragma unroll
    for (int j0 = 0; j0 < SPL; j0 += EMIT) {
      if (j0 * LPN < f) {
        int n = 0;
#pragma unroll
        for (int k = 0; k < EMIT; ++k) {
          const int j = j0 + k;
          const bool mine = j < SPL && j * LPN + sub < f;
          const uint32_t x = j < SPL ? rv[j] : 0xffffffffu;
          int rank = 0;
#pragma unroll
          for (int m = 0; m < FM; ++m) rank += (m < f && r[m] < x) ? 1 : 0;
          slot[k] = base + rank;
          u[k] = mine ? idx[o0 + x] : 0;
          n += mine ? 1 : 0;
        }
        emit_chunk(u, slot, n, b, parent, edge_src, edge_dst, visited, N, h.touched, err);
      }
    }
    return;
  }
  // Larger fan-outs (one lane per node): the subset is built in this node's
  // edge slots, then sorted.
  if (sub != 0) return;
  int32_t *r = edge_dst + base;
  for (int s = 0; s < f; ++s) {
    int64_t j = d - f + s;
    uint64_t hs = mix64(key + GAMMA * (uint64_t)(s + 1));
    int32_t tt = (int32_t)__umul64hi(hs, (uint64_t)(j + 1));
    bool seen = false;
    for (int m = 0; m < s; ++m) seen |= (r[m] == tt);
    r[s] = seen ? (int32_t)j : tt;
  }
  for (int s = 1; s < f; ++s) {  // insertion sort
    int32_t x = r[s];
    int m = s - 1;
    while (m >= 0 && r[m] > x) {
      r[m + 1] = r[m];
      --m;
    }
    r[m + 1] = x;
  }
  for (int s0 = 0; s0 < f; s0 += EMIT) {
    const int n = f - s0 < EMIT ? f - s0 : EMIT;
#pragma unroll
    for (int k = 0; k < EMIT; ++k) {
      slot[k] = base + s0 + k;
      u[k] = k < n ? idx[o0 + r[s0 + k]] : 0;
    }
    emit_chunk(u, slot, n, b, parent, edge_src, edge_dst, visited, N, h.touched, err);
  }
}

// List segments: batch b's segment starts at local index seg0[b].
struct Segs {
  int B;
  int64_t start[DG_MAX_BATCHES + 1];  // prefix of segment lengths
  int64_t seg0[DG_MAX_BATCHES];
};

// Records the local index of every node of the given list segments.
__global__ __launch_bounds__(THREADS) void k_table_insert(Segs L, const int32_t *nodes,
                                                          int64_t node_cap, LocalTable table,
                                                          uint32_t *err) {
  int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (i >= L.start[L.B]) return;
  int b = find_batch_wave(L.start, L.B, i);
  int64_t j = L.seg0[b] + (i - L.start[b]);
  if (!lt_insert(table, nodes[(int64_t)b * node_cap + j], b, j)) atomicOr(err, ERR_INTERNAL);
}

// Sampled neighbours' global IDs -> local indices through the group's
// (node, batch) hash table.
__global__ __launch_bounds__(THREADS) void k_relabel(Lists L, int64_t edge_cap, int32_t *edge_dst,
                                                     LocalTable table, int64_t N, uint32_t *err) {
  int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (i >= L.start[L.B]) return;
  int b = find_batch_wave(L.start, L.B, i);
  int64_t e = (int64_t)b * edge_cap + (i - L.start[b]);
  int32_t u = edge_dst[e];
  if (u < 0 || (int64_t)u >= N) return;  // already reported
  int64_t j = lt_find(table, u, b);
  if (j < 0) {
    atomicOr(err, ERR_INTERNAL);
    return;
  }
  edge_dst[e] = (int32_t)j;
}

// The same through the direct [N][B] table.  Every looked-up pair was written
// when its node entered the batch; the range check guards that invariant.
__global__ __launch_bounds__(THREADS) void k_relabel_direct(Lists L, int64_t edge_cap,
                                                            int32_t *edge_dst,
                                                            const int32_t *local, int64_t N,
                                                            uint32_t *err) {
  int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (i >= L.start[L.B]) return;
  int b = find_batch_wave(L.start, L.B, i);
  int64_t e = (int64_t)b * edge_cap + (i - L.start[b]);
  int32_t u = edge_dst[e];
  if (u < 0 || (int64_t)u >= N) return;  // already reported
  int32_t j = local[(int64_t)u * L.B + b];
  if (j < 0 || (int64_t)j >= L.n[b]) {
    atomicOr(err, ERR_INTERNAL);
    return;
  }
  edge_dst[e] = j;
}

// ---------------------------------------------------------------- last-hop relabelling by search
// The last hop's new nodes form one ascending segment at the end of each
// batch's list, so a last-hop edge whose neighbour is one of them gets its
// local index as the neighbour's rank in that segment; only edges into nodes
// listed earlier look the direct table up.  The last hop then writes no table
// entries at all.  Each batch's segment is copied into a padded, aligned buffer
// together with a sparse index (every S-th element); a block stages its batch's
// sparse index in LDS, searches it, and reads one S-element block of the
// segment (from L2: blocks are ordered so that all blocks of a batch run on one
// XCD).
constexpr int RL_THREADS = 512;
constexpr int RL_CHUNKS = 4;          // edge chunks per block (one staging of the index)
constexpr int RL_SPARSE_MAX = 16384;  // sparse-index entries per batch (64 KB of LDS)
constexpr int RL_S_MAX_LOG2 = 6;      // block length S = 16, 32 or 64
constexpr int RL_S_MIN_LOG2 = 4;
constexpr int64_t RL_SEGMENT_MAX = (int64_t)RL_SPARSE_MAX << RL_S_MAX_LOG2;

// edges per thread for block length 2^SLOG2 (keeps the block reads within registers)
__host__ __device__ constexpr int rl_edges(int slog2) { return slog2 <= 4 ? 4 : (slog2 == 5 ? 2 : 1); }

inline int64_t rl_segcap(int64_t node_cap) {
  return (node_cap + (1 << RL_S_MAX_LOG2) + 63) & ~(int64_t)63;
}

struct LastHop {
  int B;
  int s_log2;                           // block length S = 2^s_log2
  int32_t bstart[DG_MAX_BATCHES + 1];   // logical blocks before batch b
  int32_t m[DG_MAX_BATCHES];            // length of b's last-hop segment
  int32_t ecount[DG_MAX_BATCHES];       // b's last-hop edges
  int64_t seg0[DG_MAX_BATCHES];         // local index of the segment's first node
  int64_t e0[DG_MAX_BATCHES];           // index of b's first last-hop edge
  int64_t cstart[DG_MAX_BATCHES + 1];   // prefix of the padded segment lengths
};

// Copies each batch's last-hop segment into segbuf (row b at b*segcap), padded
// with INT32_MAX to a multiple of S, and every S-th element into sparse.
__global__ __launch_bounds__(THREADS) void k_last_segments(LastHop h, const int32_t *nodes,
                                                           int64_t node_cap, int32_t *segbuf,
                                                           int64_t segcap, int32_t *sparse) {
  const int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (i >= h.cstart[h.B]) return;
  const int b = find_batch_wave(h.cstart, h.B, i);
  const int64_t r = i - h.cstart[b];
  const int32_t v = r < h.m[b] ? nodes[(int64_t)b * node_cap + h.seg0[b] + r] : INT32_MAX;
  segbuf[(int64_t)b * segcap + r] = v;
  if ((r & ((1 << h.s_log2) - 1)) == 0) sparse[(int64_t)b * RL_SPARSE_MAX + (r >> h.s_log2)] = v;
}

template <int SLOG2>
__global__ __launch_bounds__(RL_THREADS) void k_relabel_last(LastHop h, const int32_t *segbuf,
                                                             int64_t segcap,
                                                             const int32_t *sparse,
                                                             int64_t edge_cap, int32_t *edge_dst,
                                                             const int32_t *local, int64_t N,
                                                             uint32_t *err) {
  constexpr int S = 1 << SLOG2;
  constexpr int EPT = rl_edges(SLOG2);
  constexpr int PER_CHUNK = RL_THREADS * EPT;
  extern __shared__ int32_t s_sp[];
  // Each XCD takes one contiguous run of logical blocks, i.e. whole batches, one
  // after the other.
  const int lb = (int)xcd_block(blockIdx.x, gridDim.x);
  if (lb >= h.bstart[h.B]) return;  // whole block
  int b = 0;
  while (b + 1 < h.B && h.bstart[b + 1] <= lb) ++b;
  const int R = (h.m[b] + S - 1) >> SLOG2;
  const int32_t *sp = sparse + (int64_t)b * RL_SPARSE_MAX;
  for (int i = threadIdx.x; i < R; i += RL_THREADS) s_sp[i] = sp[i];
  __syncthreads();
  int top = 1;  // highest power of two <= R (uniform)
  while (top * 2 <= R) top *= 2;
  const int64_t eend = h.e0[b] + h.ecount[b];
  int32_t *ed = edge_dst + (int64_t)b * edge_cap;
  const int32_t *seg = segbuf + (int64_t)b * segcap;
  const int B = h.B;
  const int64_t seg0 = h.seg0[b];
  for (int ch = 0; ch < RL_CHUNKS; ++ch) {
    const int64_t ebase = h.e0[b] + ((int64_t)(lb - h.bstart[b]) * RL_CHUNKS + ch) * PER_CHUNK +
                          threadIdx.x;
    if (ebase - threadIdx.x >= eend) break;  // uniform
    int32_t u[EPT];
#pragma unroll
    for (int k = 0; k < EPT; ++k) {
      const int64_t e = ebase + (int64_t)k * RL_THREADS;
      u[k] = e < eend ? ed[e] : -1;
    }
    // pos = number of sparse entries <= u: the block that may hold u is pos - 1
    int pos[EPT];
#pragma unroll
    for (int k = 0; k < EPT; ++k) pos[k] = 0;
    if (R > 0) {
      for (int step = top; step > 0; step >>= 1) {
#pragma unroll
        for (int k = 0; k < EPT; ++k)
          if (pos[k] + step <= R && s_sp[pos[k] + step - 1] <= u[k]) pos[k] += step;
      }
    }
#pragma unroll
    for (int k = 0; k < EPT; ++k) {
      const int64_t e = ebase + (int64_t)k * RL_THREADS;
      if (e >= eend || u[k] < 0 || (int64_t)u[k] >= N) continue;  // bad IDs already reported
      int c = 0;
      bool found = false;
      const int blk = pos[k] - 1;
      if (blk >= 0) {
        const uint4 *bp = reinterpret_cast<const uint4 *>(seg + ((int64_t)blk << SLOG2));
#pragma unroll
        for (int q = 0; q < S / 4; ++q) {
          const uint4 x = bp[q];
          const int32_t a0 = (int32_t)x.x, a1 = (int32_t)x.y;
          const int32_t a2 = (int32_t)x.z, a3 = (int32_t)x.w;
          c += (a0 < u[k]) + (a1 < u[k]) + (a2 < u[k]) + (a3 < u[k]);
          found |= (a0 == u[k]) | (a1 == u[k]) | (a2 == u[k]) | (a3 == u[k]);
        }
      }
      int64_t j;
      if (found) {
        j = seg0 + ((int64_t)blk << SLOG2) + c;
      } else {  // a node listed before the last hop
        j = local[(int64_t)u[k] * B + b];
        if (j < 0 || j >= seg0) {
          atomicOr(err, ERR_INTERNAL);
          continue;
        }
      }
      ed[e] = (int32_t)j;
    }
  }
}

// Host staging block (int64 entries): edge bounds, compaction totals, error word.
constexpr int ST_BOUNDS = 0;                              // [B+1]
constexpr int ST_TOTALS = ST_BOUNDS + DG_MAX_BATCHES + 1; // [B+4]
constexpr int ST_ERR = ST_TOTALS + DG_MAX_BATCHES + 4;
constexpr int ST_PTOTALS = ST_ERR + 1;                      // [B+4] packing's, fused pass
constexpr int ST_SIZE = ST_PTOTALS + DG_MAX_BATCHES + 4;

// eoff at each batch's first frontier entry (and at the end).
__global__ void k_batch_bounds(Hop h, const int64_t *f_eoff, int64_t *out) {
  int b = threadIdx.x;
  if (b <= h.B) out[b] = f_eoff[h.fstart[b]];
}

inline unsigned blocks_for(int64_t n) { return (unsigned)((n + THREADS - 1) / THREADS); }

constexpr uint32_t SAMPLE_FLAGS =
    DG_SAMPLE_LAYERED | DG_SAMPLE_DIRECT | DG_SAMPLE_EXIT_CLEAR | DG_SAMPLE_ENTRY_CLEAR;

struct SampleWs {
  uint32_t *err;
  uint64_t *visited, *prev;
  uint8_t *plines;  // lines of prev that hold a bit (a byte per 8 nodes)
  int64_t *f_off, *f_deg, *f_cnt, *f_eoff, *tiles;
  LocalTable table;  // hash relabelling
  int32_t *local;    // direct relabelling: [N][B]
  int32_t *segbuf;   // direct relabelling: last-hop segments, [B][rl_segcap(node_cap)]
  int32_t *sparse;   // ... and their sparse indices, [B][RL_SPARSE_MAX]
  uint8_t *touched;  // touched marks (a byte per 2^MC_TOUCH_SHIFT nodes)
  int64_t *small;    // staging for a few counts
  MaskScan ms;
};

void carve_sample(SampleWs &w, Carve &c, int64_t N, int B, int64_t node_cap, bool direct) {
  int64_t fmax = (int64_t)B * node_cap;  // frontier entries never exceed the node lists
  w.err = c.take<uint32_t>(64);
  w.visited = c.take<uint64_t>((size_t)N);
  w.prev = c.take<uint64_t>((size_t)N);
  w.plines = c.take<uint8_t>((size_t)mc_touch_bytes(N));
  w.f_off = c.take<int64_t>((size_t)fmax);
  w.f_deg = c.take<int64_t>((size_t)fmax);
  w.f_cnt = c.take<int64_t>((size_t)fmax);
  w.f_eoff = c.take<int64_t>((size_t)fmax + 1);
  w.tiles = c.take<int64_t>(scan_tile_count(fmax));
  w.table.bits = direct ? 0 : lt_bits_for(fmax);
  w.table.slots = direct ? nullptr : c.take<uint64_t>((size_t)1 << w.table.bits);
  w.local = direct ? c.take<int32_t>((size_t)N * (size_t)B) : nullptr;
  w.segbuf = direct ? c.take<int32_t>((size_t)B * (size_t)rl_segcap(node_cap)) : nullptr;
  w.sparse = direct ? c.take<int32_t>((size_t)B * RL_SPARSE_MAX) : nullptr;
  w.touched = c.take<uint8_t>((size_t)mc_touch_bytes(N));
  w.small = c.take<int64_t>(ST_SIZE);
  w.ms = MaskScan{};
  w.ms.N = N;
  w.ms.B = B;
  mask_scan_carve(w.ms, c);
}

int check_err(uint32_t *err_dev, hipStream_t s) {
  uint32_t bits = 0;
  DG_TRY(read_to_host(&bits, err_dev, sizeof(bits), s));
  if (bits) return set_error(DG_EINVAL, "invalid input data: %s", describe_device_error(bits));
  return DG_OK;
}

}  // namespace
}  // namespace dg

using namespace dg;

extern "C" int dg_sample_bounds(int64_t num_nodes, int64_t num_edges, int32_t S,
                                const int32_t *fanouts, int32_t K, uint32_t flags,
                                int64_t *node_cap, int64_t *edge_cap) {
  if (!node_cap || !edge_cap || (K > 0 && !fanouts) || S < 1 || K < 0 || num_nodes < 1 ||
      num_edges < 0 || (flags & ~SAMPLE_FLAGS))
    return set_error(DG_EINVAL, "dg_sample_bounds: bad argument");
  const bool layered = flags & DG_SAMPLE_LAYERED;
  // Saturating arithmetic: once a count reaches its graph bound it stays there.
  // n = nodes so far, front = nodes that sample at the next hop; per hop the
  // edges are distinct CSR edges (each frontier node samples once), so a hop
  // adds at most min(f * front, E) edges.
  const int64_t big = INT64_MAX / 4;
  int64_t n = S, e = 0, front = S;
  for (int k = 0; k < K; ++k) {
    const int32_t f = fanouts[k];
    int64_t hop_e = f < 0 ? num_edges : (front > big / (f > 0 ? f : 1) ? big : front * f);
    if (hop_e > num_edges) hop_e = num_edges;
    e = e > big - hop_e ? big : e + hop_e;
    const int64_t grown = n > big - hop_e ? big : n + hop_e;
    front = layered ? (grown < num_nodes ? grown : num_nodes) : hop_e;
    n = grown < num_nodes ? grown : num_nodes;
    if (front > num_nodes) front = num_nodes;
  }
  // without layering a node samples at most once, so a batch's edges are
  // distinct CSR edges
  if (!layered && e > num_edges) e = num_edges;
  *node_cap = n;
  *edge_cap = e < 1 ? 1 : e;
  return DG_OK;
}

extern "C" size_t dg_sample_workspace_bytes(int64_t num_nodes, int32_t B, int64_t node_cap,
                                            int64_t edge_cap, uint32_t flags) {
  (void)edge_cap;
  if (num_nodes < 1 || B < 1 || B > DG_MAX_BATCHES || node_cap < 1 || (flags & ~SAMPLE_FLAGS))
    return 0;
  Carve c(nullptr);
  SampleWs w;
  carve_sample(w, c, num_nodes, B, node_cap, (flags & DG_SAMPLE_DIRECT) != 0);
  return c.used;
}

namespace dg {
namespace {

// Event indices of a sampling call's phases (read once the call's work is done).
struct SampleMarks {
  int start = -1, r0 = -1, r1 = -1, nhop = 0;
  int hop[8][3];
};

// Packing state of dg_sample_pack_group, carved from its packing workspace:
// what the fused last hop writes besides sampling's outputs, and what it
// reports back.
struct PackInto {
  PackWs pw;          // packing's workspace (last in the carve, see carve_sample_pack)
  size_t pw_offset;   // its offset in the packing workspace
  uint64_t *pinfo;    // [pinfo_cap] node and list slot of each packed pair (fused pass)
  int64_t pinfo_cap;
  int32_t *cw_slot;   // the fused pass's cache slot per listed word
  uint8_t *lines;     // member lines, for a group packed by packing's own passes
  int64_t unc_cap, pair_cap;
  int64_t *packed_ptr;
  int64_t packed_cap;
  int32_t *group_unique;
  int64_t unique_cap;
  // set by sample_impl
  bool fused = false;                 // the last hop's compaction did packing's pass
  int64_t ptot[DG_MAX_BATCHES + 4];  // packing's row totals (fused)
  uint32_t *err = nullptr;            // sampling's device error word, not yet checked
  uint64_t *visited = nullptr;        // the membership words sampling used
  int32_t *local = nullptr;           // the direct table (DG_SAMPLE_DIRECT)
};

void carve_sample_pack(PackInto &pk, Carve &c, int64_t N, int B, int64_t node_cap) {
  const int64_t total = (int64_t)B * node_cap;
  pk.pinfo = c.take<uint64_t>((size_t)total);
  pk.pinfo_cap = total;
  pk.cw_slot = c.take<int32_t>((size_t)mc_blocks(N) * MC_BLOCK_NODES);
  pk.lines = c.take<uint8_t>((size_t)mc_touch_bytes(N));
  pk.pw_offset = c.used;  // packing's own workspace last: the unfused path hands it on whole
  carve_pack(pk.pw, c, N, B, total);
  pk.unc_cap = (total < N ? total : N) + 1;
  pk.pair_cap = total + 1;
}

int sample_impl(const dg_csr *g, const int32_t *seeds, int32_t B, int32_t S, int64_t batch_base,
                const int32_t *fanouts, int32_t K, uint64_t rng_seed, uint32_t flags,
                int64_t node_cap, int32_t *nodes, int64_t *hop_ptr, int64_t edge_cap,
                int32_t *edge_src, int32_t *edge_dst, int64_t *edge_ptr, uint64_t *membership,
                uint8_t *member_lines, const int32_t *cache_slot, int32_t *loc, void *ws,
                size_t ws_bytes, hipStream_t stream, dg_sizes *sizes, PhaseTimer &tm,
                SampleMarks &mk, PackInto *pk) {
  if (!g || !seeds || !nodes || !hop_ptr || !edge_src || !edge_dst || !edge_ptr || !sizes ||
      (K > 0 && !fanouts))
    return set_error(DG_EINVAL, "dg_sample_group: null pointer argument");
  if (!cache_slot != !loc)
    return set_error(DG_EINVAL, "dg_sample_group: cache_slot and loc go together");
  if (!g->offsets || (g->num_edges > 0 && !g->indices) || g->num_nodes < 1 ||
      g->num_nodes > 0x7fffffffll || g->num_edges < 0)
    return set_error(DG_EINVAL, "dg_sample_group: bad CSR description");
  if (flags & ~SAMPLE_FLAGS)
    return set_error(DG_EINVAL, "dg_sample_group: unknown flags 0x%x", flags);
  const bool layered = flags & DG_SAMPLE_LAYERED;
  const bool direct = flags & DG_SAMPLE_DIRECT;
  const bool entry_clear = flags & DG_SAMPLE_ENTRY_CLEAR;
  const bool exit_clear = flags & DG_SAMPLE_EXIT_CLEAR;
  if (entry_clear && !membership)
    return set_error(DG_EINVAL, "dg_sample_group: DG_SAMPLE_ENTRY_CLEAR needs membership");
  if (B < 1 || B > DG_MAX_BATCHES || S < 1 || K < 0 || node_cap < S || edge_cap < 0 ||
      (int64_t)S > g->num_nodes)
    return set_error(DG_EINVAL, "dg_sample_group: bad sizes (B=%d S=%d K=%d node_cap=%lld)", B,
                     S, K, (long long)node_cap);
  if (node_cap > LT_MAX_VALUE)
    return set_error(DG_EINVAL, "dg_sample_group: node_cap above 2^27 - 1 is not supported");
  const size_t need_ws = dg_sample_workspace_bytes(g->num_nodes, B, node_cap, edge_cap, flags);
  if (!ws || ws_bytes < need_ws || ((uintptr_t)ws & 255))
    return set_error(DG_EWORKSPACE, "dg_sample_group: workspace needs %zu bytes, 256-aligned",
                     need_ws);

  const int64_t N = g->num_nodes, E = g->num_edges;
  hipStream_t s = stream;
  SampleWs w;
  Carve c(ws);
  carve_sample(w, c, N, B, node_cap, direct);
  w.ms.err = w.err;

  memset(sizes, 0, sizeof(*sizes));
  sizes->packed_rows = sizes->unique_nodes = sizes->unique_packed = -1;
  sizes->exact = 1;
  mk.nhop = 0;
  mk.start = tm.mark();

  int rc;
  if ((rc = fill_u64(reinterpret_cast<uint64_t *>(w.err), 32, 0, s))) return rc;
  if (membership) w.visited = membership;
  // prev (workspace) and visited must start all-zero: cleared here unless the
  // caller asserts that they already are (see DG_SAMPLE_ENTRY_CLEAR)
  if (!entry_clear) {
    if ((rc = fill_u64(w.visited, (size_t)N, 0, s))) return rc;
    if ((rc = fill_u64(w.prev, (size_t)N, 0, s))) return rc;
    if ((rc = fill_u64(reinterpret_cast<uint64_t *>(w.plines), (size_t)mc_touch_bytes(N) / 8, 0,
                       s)))
      return rc;
  }
  bool prev_cleared = false;  // the last hop's count pass zeroed prev
  bool lines_done = false;    // the last hop's count pass wrote member_lines
  bool rl_search = false;     // the last hop's edges are relabelled by search
  hipLaunchKernelGGL(k_seed_init, dim3(blocks_for((int64_t)B * S)), dim3(THREADS), 0, s, seeds,
                     B, S, N, node_cap, nodes, w.visited, w.prev, w.plines, w.local, cache_slot,
                     loc,
                     w.err);
  DG_HIP(hipGetLastError());  // bad seeds are reported at the first hop's round trip

  int64_t n_b[DG_MAX_BATCHES], e_b[DG_MAX_BATCHES];
  for (int b = 0; b < B; ++b) {
    n_b[b] = S;
    e_b[b] = 0;
    hop_ptr[(int64_t)b * (K + 2) + 0] = 0;
    hop_ptr[(int64_t)b * (K + 2) + 1] = S;
  }

  Hop h;
  memset(&h, 0, sizeof(h));
  h.B = B;
  for (int b = 0; b < B; ++b)
    h.bstate[b] = mix64(rng_seed + GAMMA * ((uint64_t)(batch_base + b) + 1ull));
  int64_t fbeg[DG_MAX_BATCHES], fend[DG_MAX_BATCHES];
  for (int b = 0; b < B; ++b) {
    fbeg[b] = 0;
    fend[b] = S;
  }
  for (int k = 1; k <= K; ++k) {
    for (int b = 0; b < B; ++b) edge_ptr[(int64_t)b * (K + 1) + (k - 1)] = e_b[b];
    const int32_t f = fanouts[k - 1];
    h.f = f;
    h.k = k;
    h.fstart[0] = 0;
    for (int b = 0; b < B; ++b) {
      h.fpos[b] = fbeg[b];
      h.fstart[b + 1] = h.fstart[b] + (fend[b] - fbeg[b]);
      h.ebase[b] = e_b[b];
    }
    h.ftot = h.fstart[B];
    int64_t new_b[DG_MAX_BATCHES];
    if (h.ftot == 0 || f == 0) {
      for (int b = 0; b < B; ++b) new_b[b] = 0;
    } else {
      const int ev0 = tm.mark();
      // A hop whose edges can reach at most N/16 nodes marks the mask lines it
      // touches (a byte store per edge), and its count pass reads only those.
      // On larger hops the stores cost more time than the lines they spare.
      // The last hop never marks when the call must write the member-lines map
      // or leave prev clear: its count pass then reads every word anyway and
      // does both on the way, where marks would need a pass over the whole mask
      // for the map and a fill of prev afterwards.
      const int64_t ebound = f < 0 ? E : h.ftot * (int64_t)f;
      // With a packing state (and the direct table, which gives older pairs'
      // list slots) the last hop's compaction also does packing's pass.
      const bool fuse = pk && direct && k == K;
      const bool full_last = k == K && (member_lines || exit_clear || fuse);
      h.touched = (ebound <= N / 16 && !full_last) ? w.touched : nullptr;
      if (h.touched && (rc = fill_u64(reinterpret_cast<uint64_t *>(w.touched),
                                      (size_t)mc_touch_bytes(N) / 8, 0, s)))
        return rc;
      hipLaunchKernelGGL(k_frontier_degree, dim3(blocks_for(h.ftot)), dim3(THREADS), 0, s, h,
                         nodes, node_cap, g->offsets, N, E, w.f_off, w.f_deg, w.f_cnt, w.err);
      DG_HIP(hipGetLastError());
      if ((rc = scan_exclusive(w.f_cnt, w.f_eoff, h.ftot, w.tiles, s))) return rc;
      // edge offsets at the batch boundaries, kept on the device
      hipLaunchKernelGGL(k_batch_bounds, dim3(1), dim3(DG_MAX_BATCHES + 1), 0, s, h, w.f_eoff,
                         w.small + ST_BOUNDS);
      // lanes per frontier node: up to 8 while the frontier has fewer than 2^20
      // entries (never more lanes than draws; fan-outs above FMAX keep one)
      int lpn = 1;
      while (lpn < 8 && h.ftot * lpn < (1 << 20) && (f < 0 || (f <= FMAX && 2 * lpn <= f)))
        lpn *= 2;
      const dim3 hg(blocks_for(h.ftot * lpn)), hb(THREADS);
      // register-path capacity: the smallest that holds f (8 when f does not
      // take the register path at all)
      const int fm = (f < 0 || f > FMAX || f <= 8) ? 8 : (f <= 16 ? 16 : 32);
      auto launch = [&](auto lpn_c, auto fm_c) {
        hipLaunchKernelGGL((k_hop_sample<decltype(lpn_c)::value, decltype(fm_c)::value>), hg, hb,
                           0, s, h, nodes, node_cap, g->indices, w.f_off, w.f_deg, w.f_eoff,
                           w.small + ST_BOUNDS, edge_cap, edge_src, edge_dst, w.visited, N,
                           w.err);
      };
      auto launch_fm = [&](auto lpn_c) {
        if (fm == 8) launch(lpn_c, std::integral_constant<int, 8>());
        else if (fm == 16) launch(lpn_c, std::integral_constant<int, 16>());
        else launch(lpn_c, std::integral_constant<int, 32>());
      };
      if (lpn == 8) launch_fm(std::integral_constant<int, 8>());
      else if (lpn == 4) launch_fm(std::integral_constant<int, 4>());
      else if (lpn == 2) launch_fm(std::integral_constant<int, 2>());
      else launch_fm(std::integral_constant<int, 1>());
      DG_HIP(hipGetLastError());
      const int ev1 = tm.mark();
      // new nodes of this hop, per batch, ascending; the write pass needs only
      // the list starts known before the hop, so it is queued before the host
      // reads this hop's counts (it stops at each list's capacity)
      w.ms.mask = w.visited;
      w.ms.prev = w.prev;
      w.ms.plines = w.plines;
      w.ms.keep_prev = k < K;  // after the last hop nothing reads prev
      w.ms.touched = h.touched;
      // With DG_SAMPLE_EXIT_CLEAR the last hop's count pass zeroes every prev
      // word it reads; that is all non-zero ones (prev is a subset of visited)
      // unless touched marks leave some lines unread.
      w.ms.clear_prev = exit_clear && k == K && !h.touched;
      prev_cleared = w.ms.clear_prev;
      // the last hop's count pass reads every word unless touched marks limit it
      w.ms.lines_out = (member_lines && k == K && !h.touched) ? member_lines : nullptr;
      lines_done = w.ms.lines_out != nullptr;
      w.ms.cache_slot = nullptr;
      w.ms.totals = w.small + ST_TOTALS;
      w.ms.err_stage = w.small + ST_ERR;
      FuseScan F;
      if (fuse) {
        MaskScan &vp = pk->pw.ms;
        vp.totals = w.small + ST_PTOTALS;
        vp.err_stage = nullptr;
        vp.err = w.err;
        memset(&F, 0, sizeof(F));
        F.mask = w.visited;
        F.prev = w.prev;
        F.plines = w.plines;
        F.cache_slot = cache_slot;
        F.N = N;
        F.B = B;
        F.nblk = w.ms.nblk;
        F.clear_prev = w.ms.clear_prev;
        F.err = w.err;
        F.wcnt = w.ms.wcnt;
        F.cw_mask = w.ms.cw_mask;
        F.cw_new = vp.cw_mask;
        F.cw_off = w.ms.cw_off;
        F.cw_slot = pk->cw_slot;
        F.cnt_s = w.ms.cnt;
        F.wpre_s = w.ms.wpre;
        F.cnt_p = vp.cnt;
        F.wpre_p = vp.wpre;
        F.base_s = w.ms.base;
        F.base_p = vp.base;
        w.ms.lines_out = nullptr;
        lines_done = false;
        if ((rc = fuse_scan_count(F, w.ms, vp, s))) return rc;
      } else if ((rc = mask_scan_count(w.ms, s))) {
        return rc;
      }
      for (int b = 0; b < B; ++b) {
        w.ms.seg_base[b] = (int64_t)b * node_cap + n_b[b];
        w.ms.seg_end[b] = (int64_t)(b + 1) * node_cap;
        w.ms.local_base[b] = n_b[b];
      }
      // Direct relabelling: the last hop's edges find their new neighbours by
      // search in the hop's segment, so that hop writes no table entries,
      // unless a segment could outgrow the sparse index (an upper bound is all
      // that is known before the hop's counts come back).
      if (direct && k == K) {
        int64_t mbound = 0, ebound = 0;
        for (int b = 0; b < B; ++b) {
          const int64_t front = h.fstart[b + 1] - h.fstart[b];
          int64_t mb = node_cap - n_b[b];
          const int64_t eb = f < 0 ? E : (front > E / (f > 0 ? f : 1) ? E : front * f);
          if (eb < mb) mb = eb;
          if (N < mb) mb = N;
          if (mb > mbound) mbound = mb;
          if (eb > ebound) ebound = eb;
        }
        rl_search = mbound <= RL_SEGMENT_MAX && ebound <= INT32_MAX;
      }
      w.ms.seg_out = nodes;
      w.ms.local_out = (k == K && rl_search) ? nullptr : w.local;
      w.ms.loc_slot = cache_slot;  // the list's address-table entries beside it
      w.ms.loc_out = loc;
      w.ms.uniq_out = nullptr;
      w.ms.unc_ids = nullptr;
      w.ms.unc_off = nullptr;
      w.ms.nodeoff = nullptr;
      w.ms.pairdest = nullptr;
      if (fuse) {
        F.node_cap = node_cap;
        for (int b = 0; b < B; ++b) {
          F.seg_base[b] = w.ms.seg_base[b];
          F.seg_end[b] = w.ms.seg_end[b];
        }
        F.seg_out = nodes;
        F.loc_out = loc;
        F.local_out = w.ms.local_out;
        F.packed_ptr = pk->packed_ptr;
        F.packed_cap = pk->packed_cap < pk->pinfo_cap ? pk->packed_cap : pk->pinfo_cap;
        F.pinfo = pk->pinfo;
        F.uniq_out = pk->group_unique;
        F.unique_cap = pk->unique_cap;
        F.unc_ids = pk->pw.unc_ids;
        F.unc_off = pk->pw.unc_off;
        F.unc_cap = pk->unc_cap;
        F.nodeoff = nullptr;  // the address tables come from pinfo
        F.pairdest = pk->pw.pairdest;
        F.pair_cap = pk->pair_cap;
        if ((rc = fuse_scan_write(F, w.small + ST_PTOTALS, pk->packed_ptr, s))) return rc;
      } else if ((rc = mask_scan_write(w.ms, s))) {
        return rc;
      }
      const int ev2 = tm.mark();
      // one round trip per hop: edge bounds, node counts and the error word
      // (and packing's totals after a fused pass)
      int64_t st[ST_SIZE];
      DG_TRY(read_to_host(st, w.small, sizeof(int64_t) * (fuse ? ST_SIZE : ST_PTOTALS), s));
      if (st[ST_ERR])
        return set_error(DG_EINVAL, "invalid input data: %s",
                         describe_device_error((uint32_t)st[ST_ERR]));
      const int64_t *bound = st + ST_BOUNDS;
      bool over = false, nover = false;
      for (int b = 0; b < B; ++b) {
        const int64_t cnt = bound[b + 1] - bound[b];
        new_b[b] = st[ST_TOTALS + b];
        if (e_b[b] + cnt > edge_cap) over = true;
        if (n_b[b] + new_b[b] > node_cap) nover = true;
        if (e_b[b] + cnt > sizes->max_batch_edges) sizes->max_batch_edges = e_b[b] + cnt;
        e_b[b] += cnt;
      }
      if (over) {  // the node counts of this hop are not meaningful
        sizes->exact = 0;
        for (int b = 0; b < B; ++b)
          if (n_b[b] > sizes->max_batch_nodes) sizes->max_batch_nodes = n_b[b];
        return set_error(DG_ECAPACITY, "dg_sample_group: edge_cap %lld too small at hop %d",
                         (long long)edge_cap, k);
      }
      for (int b = 0; b < B; ++b)
        if (n_b[b] + new_b[b] > sizes->max_batch_nodes) sizes->max_batch_nodes = n_b[b] + new_b[b];
      if (nover) {
        sizes->exact = 0;
        return set_error(DG_ECAPACITY, "dg_sample_group: node_cap %lld too small at hop %d",
                         (long long)node_cap, k);
      }
      if (fuse) {
        pk->fused = true;
        for (int r = 0; r < mc_rows(B); ++r) pk->ptot[r] = st[ST_PTOTALS + r];
      }
      if (mk.nhop < 8) {
        mk.hop[mk.nhop][0] = ev0;
        mk.hop[mk.nhop][1] = ev1;
        mk.hop[mk.nhop][2] = ev2;
        ++mk.nhop;
      }
    }
    for (int b = 0; b < B; ++b) {
      // next frontier: the nodes new at this hop, or (layered) every node so far
      fbeg[b] = layered ? 0 : n_b[b];
      n_b[b] += new_b[b];
      fend[b] = n_b[b];
      hop_ptr[(int64_t)b * (K + 2) + k + 1] = n_b[b];
    }
  }
  for (int b = 0; b < B; ++b) edge_ptr[(int64_t)b * (K + 1) + K] = e_b[b];

  // Local IDs through the (node, batch) table.
  mk.r0 = tm.mark();
  Lists LE;
  LE.B = B;
  LE.start[0] = 0;
  for (int b = 0; b < B; ++b) {
    LE.start[b + 1] = LE.start[b] + e_b[b];
    LE.n[b] = n_b[b];
  }
  if (LE.start[B] > 0 && direct && rl_search) {
    // edges of the hops before the last through the table, the last hop's by
    // search in its segment
    LastHop lh;
    memset(&lh, 0, sizeof(lh));
    lh.B = B;
    int64_t m_max = 0;
    for (int b = 0; b < B; ++b) {
      const int64_t before = edge_ptr[(int64_t)b * (K + 1) + (K - 1)];
      LE.start[b + 1] = LE.start[b] + before;
      lh.seg0[b] = hop_ptr[(int64_t)b * (K + 2) + K];
      lh.m[b] = (int32_t)(n_b[b] - lh.seg0[b]);
      lh.e0[b] = before;
      lh.ecount[b] = (int32_t)(e_b[b] - before);
      if (lh.m[b] > m_max) m_max = lh.m[b];
    }
    lh.s_log2 = RL_S_MIN_LOG2;
    while (lh.s_log2 < RL_S_MAX_LOG2 && (m_max + (1 << lh.s_log2) - 1) >> lh.s_log2 > RL_SPARSE_MAX)
      ++lh.s_log2;
    const int S = 1 << lh.s_log2;
    const int per_block = RL_THREADS * rl_edges(lh.s_log2) * RL_CHUNKS;
    lh.cstart[0] = 0;
    lh.bstart[0] = 0;
    int64_t r_max = 0;
    for (int b = 0; b < B; ++b) {
      const int64_t r = (lh.m[b] + S - 1) / S;
      if (r > r_max) r_max = r;
      lh.cstart[b + 1] = lh.cstart[b] + r * S;
      lh.bstart[b + 1] = lh.bstart[b] + (int32_t)((lh.ecount[b] + per_block - 1) / per_block);
    }
    if (r_max > RL_SPARSE_MAX)
      return set_error(DG_EINVAL, "internal: last-hop segment of %lld nodes", (long long)m_max);
    if (LE.start[B] > 0) {
      hipLaunchKernelGGL(k_relabel_direct, dim3(blocks_for(LE.start[B])), dim3(THREADS), 0, s,
                         LE, edge_cap, edge_dst, w.local, N, w.err);
    }
    if (lh.cstart[B] > 0)
      hipLaunchKernelGGL(k_last_segments, dim3(blocks_for(lh.cstart[B])), dim3(THREADS), 0, s,
                         lh, nodes, node_cap, w.segbuf, rl_segcap(node_cap), w.sparse);
    if (lh.bstart[B] > 0) {
      const unsigned grid = (unsigned)((lh.bstart[B] + 7) & ~7);
      const size_t lds = (size_t)(r_max > 0 ? r_max : 1) * sizeof(int32_t);
      auto go = [&](auto slog2) {
        hipLaunchKernelGGL((k_relabel_last<decltype(slog2)::value>), dim3(grid),
                           dim3(RL_THREADS), lds, s, lh, w.segbuf, rl_segcap(node_cap),
                           w.sparse, edge_cap, edge_dst, w.local, N, w.err);
      };
      if (lh.s_log2 == 4) go(std::integral_constant<int, 4>());
      else if (lh.s_log2 == 5) go(std::integral_constant<int, 5>());
      else go(std::integral_constant<int, 6>());
    }
    DG_HIP(hipGetLastError());
  } else if (LE.start[B] > 0 && direct) {
    hipLaunchKernelGGL(k_relabel_direct, dim3(blocks_for(LE.start[B])), dim3(THREADS), 0, s, LE,
                       edge_cap, edge_dst, w.local, N, w.err);
    DG_HIP(hipGetLastError());
  } else if (LE.start[B] > 0) {
    // the table holds every (node, batch) pair of the group, at load <= 1/2
    Segs LS;
    LS.B = B;
    LS.start[0] = 0;
    for (int b = 0; b < B; ++b) {
      LS.start[b + 1] = LS.start[b] + n_b[b];
      LS.seg0[b] = 0;
    }
    LocalTable table = w.table;
    table.bits = lt_bits_for(LS.start[B]);
    if ((rc = fill_u64(table.slots, (size_t)1 << table.bits, 0, s))) return rc;
    hipLaunchKernelGGL(k_table_insert, dim3(blocks_for(LS.start[B])), dim3(THREADS), 0, s, LS,
                       nodes, node_cap, table, w.err);
    hipLaunchKernelGGL(k_relabel, dim3(blocks_for(LE.start[B])), dim3(THREADS), 0, s, LE,
                       edge_cap, edge_dst, table, N, w.err);
    DG_HIP(hipGetLastError());
  }
  mk.r1 = tm.mark();
  if (exit_clear && !prev_cleared &&
      ((rc = fill_u64(w.prev, (size_t)N, 0, s)) ||
       (rc = fill_u64(reinterpret_cast<uint64_t *>(w.plines), (size_t)mc_touch_bytes(N) / 8, 0,
                      s))))
    return rc;
  if (member_lines && !lines_done && !(pk && pk->fused) &&
      (rc = member_lines_pass(w.visited, N, B, member_lines, s)))
    return rc;
  if (pk) {  // the caller checks the error word after its own work
    pk->err = w.err;
    pk->visited = w.visited;
    pk->local = w.local;
  } else if ((rc = check_err(w.err, s))) {
    return rc;
  }

  int64_t tn = 0, te = 0, mn = 0, me = 0;
  for (int b = 0; b < B; ++b) {
    tn += n_b[b];
    te += e_b[b];
    if (n_b[b] > mn) mn = n_b[b];
    if (e_b[b] > me) me = e_b[b];
  }
  sizes->max_batch_nodes = mn;
  sizes->max_batch_edges = me;
  sizes->total_nodes = tn;
  sizes->total_edges = te;
  return DG_OK;
}

// Sampling's phase times from the marks of a finished call.
void sample_times(const PhaseTimer &tm, const SampleMarks &mk, dg_timing *timing) {
  float t_sample = 0.f, t_dedup = 0.f;
  for (int i = 0; i < mk.nhop && i < 8; ++i) {
    t_sample += tm.ms(mk.hop[i][0], mk.hop[i][1]);
    t_dedup += tm.ms(mk.hop[i][1], mk.hop[i][2]);
  }
  timing->sample_ms = t_sample;
  timing->dedup_ms = t_dedup;
  timing->relabel_ms = tm.ms(mk.r0, mk.r1);
  timing->total_ms = tm.ms(mk.start, mk.r1);
}

}  // namespace
}  // namespace dg

extern "C" int dg_sample_group(const dg_csr *g, const int32_t *seeds, int32_t B, int32_t S,
                               int64_t batch_base, const int32_t *fanouts, int32_t K,
                               uint64_t rng_seed, uint32_t flags, int64_t node_cap,
                               int32_t *nodes,
                               int64_t *hop_ptr, int64_t edge_cap, int32_t *edge_src,
                               int32_t *edge_dst, int64_t *edge_ptr, uint64_t *membership,
                               uint8_t *member_lines, const int32_t *cache_slot, int32_t *loc,
                               void *ws, size_t ws_bytes, hipStream_t stream, dg_sizes *sizes,
                               dg_timing *timing) {
  if (timing) memset(timing, 0, sizeof(*timing));
  PhaseTimer tm(timing != nullptr, stream);
  SampleMarks mk;
  const int rc = sample_impl(g, seeds, B, S, batch_base, fanouts, K, rng_seed, flags, node_cap,
                             nodes, hop_ptr, edge_cap, edge_src, edge_dst, edge_ptr, membership,
                             member_lines, cache_slot, loc, ws, ws_bytes, stream, sizes, tm, mk,
                             nullptr);
  if (rc == DG_OK && timing) sample_times(tm, mk, timing);
  return rc;
}

extern "C" size_t dg_sample_pack_workspace_bytes(int64_t num_nodes, int32_t B,
                                                 int64_t node_cap) {
  if (num_nodes < 1 || B < 1 || B > DG_MAX_BATCHES || node_cap < 1 ||
      node_cap > INT64_MAX / DG_MAX_BATCHES)
    return 0;
  Carve c(nullptr);
  PackInto pk;
  carve_sample_pack(pk, c, num_nodes, B, node_cap);
  return c.used;
}

extern "C" int dg_sample_pack_group(
    const dg_csr *g, const int32_t *seeds, int32_t B, int32_t S, int64_t batch_base,
    const int32_t *fanouts, int32_t K, uint64_t rng_seed, uint32_t flags, int64_t node_cap,
    int32_t *nodes, int64_t *hop_ptr, int64_t edge_cap, int32_t *edge_src, int32_t *edge_dst,
    int64_t *edge_ptr, uint64_t *membership, const int32_t *cache_slot, int32_t *loc,
    const void *feats, int64_t row_bytes, int64_t packed_cap, void *packed, int32_t *packed_ids,
    int64_t *packed_ptr, int64_t *packed_ptr_host, int32_t *group_unique, int64_t unique_cap,
    uint32_t pack_flags, void *ws, size_t ws_bytes, void *pack_ws, size_t pack_ws_bytes,
    hipStream_t stream, hipStream_t rows_stream, dg_sizes *sizes, dg_timing *timing) {
  if (!g || !cache_slot || !loc || !feats || !packed_ptr || !packed_ptr_host || !sizes ||
      !hop_ptr)
    return set_error(DG_EINVAL, "dg_sample_pack_group: null pointer argument");
  if (row_bytes < 1 || packed_cap < 0 || unique_cap < 0 || (packed_cap > 0 && !packed_ids))
    return set_error(DG_EINVAL, "dg_sample_pack_group: bad packing sizes");
  if (pack_flags & ~DG_PACK_ROWS_STREAM)
    return set_error(DG_EINVAL, "dg_sample_pack_group: unknown pack flags 0x%x", pack_flags);
  if ((pack_flags & DG_PACK_ROWS_STREAM) && timing)
    return set_error(DG_EINVAL, "dg_sample_pack_group: timing cannot be combined with "
                                "DG_PACK_ROWS_STREAM");
  const size_t need = dg_sample_pack_workspace_bytes(g->num_nodes, B, node_cap);
  if (need == 0 || K < 0)
    return set_error(DG_EINVAL, "dg_sample_pack_group: bad sizes (B=%d K=%d node_cap=%lld)", B,
                     K, (long long)node_cap);
  if (!pack_ws || pack_ws_bytes < need || ((uintptr_t)pack_ws & 255))
    return set_error(DG_EWORKSPACE,
                     "dg_sample_pack_group: packing workspace needs %zu bytes, 256-aligned",
                     need);
  const bool rows_async = (pack_flags & DG_PACK_ROWS_STREAM) && packed;
  const int64_t N = g->num_nodes;
  PackInto pk;
  Carve c(pack_ws);
  carve_sample_pack(pk, c, N, B, node_cap);
  pk.packed_ptr = packed_ptr;
  pk.packed_cap = packed_cap;
  pk.group_unique = group_unique;
  pk.unique_cap = group_unique ? unique_cap : 0;
  if (timing) memset(timing, 0, sizeof(*timing));
  PhaseTimer tm(timing != nullptr, stream);
  SampleMarks mk;
  int rc = sample_impl(g, seeds, B, S, batch_base, fanouts, K, rng_seed, flags, node_cap, nodes,
                       hop_ptr, edge_cap, edge_src, edge_dst, edge_ptr, membership, pk.lines,
                       cache_slot, loc, ws, ws_bytes, stream, sizes, tm, mk, &pk);
  if (rc) return rc;
  int64_t n_b[DG_MAX_BATCHES];
  for (int b = 0; b < B; ++b) n_b[b] = hop_ptr[(int64_t)b * (K + 2) + K + 1];

  if (!pk.fused) {
    // No fused pass (hash relabelling, or a last hop with nothing to sample):
    // packing's own passes over the lists sampling wrote.
    if ((rc = check_err(pk.err, stream))) return rc;
    if (timing) sample_times(tm, mk, timing);
    dg_sizes ps;
    dg_timing pt;
    rc = pack_impl(feats, N, row_bytes, cache_slot, B, nodes, node_cap, n_b, packed_cap, packed,
                   packed_ids, packed_ptr, packed_ptr_host, loc, group_unique, unique_cap,
                   membership ? membership : pk.visited, pk.lines, nullptr, 0, nullptr,
                   DG_PACK_CLEAR_MEMBERSHIP | DG_PACK_LOC_PENDING |
                       (pack_flags & DG_PACK_ROWS_STREAM),
                   static_cast<char *>(pack_ws) + pk.pw_offset, pack_ws_bytes - pk.pw_offset,
                   stream, rows_stream, &ps, timing ? &pt : nullptr, false);
    sizes->packed_rows = ps.packed_rows;
    sizes->unique_nodes = ps.unique_nodes;
    sizes->unique_packed = ps.unique_packed;
    if (rc) return rc;
    if (timing) {
      timing->mark_ms = pt.mark_ms;
      timing->order_ms = pt.order_ms;
      timing->loc_ms = pt.loc_ms;
      timing->gather_ms = pt.gather_ms;
      timing->total_ms += pt.total_ms;
    }
    return DG_OK;
  }

  // Packing's sizes came back with the last hop's counts.
  int64_t rows = 0;
  packed_ptr_host[0] = 0;
  for (int b = 0; b < B; ++b) {
    rows += pk.ptot[b];
    packed_ptr_host[b + 1] = rows;
  }
  sizes->packed_rows = rows;
  sizes->unique_nodes = pk.ptot[row_all(B)];
  sizes->unique_packed = pk.ptot[row_packed(B)];
  if (rows != pk.ptot[row_pairs(B)] || pk.ptot[row_all_pairs(B)] != sizes->total_nodes)
    return set_error(DG_EINVAL, "dg_sample_pack_group: internal pair count mismatch");
  if (rows > packed_cap || (group_unique && sizes->unique_nodes > unique_cap))
    return set_error(DG_ECAPACITY,
                     "dg_sample_pack_group: need packed_cap >= %lld and unique_cap >= %lld",
                     (long long)rows, (long long)sizes->unique_nodes);
  FusedTail t;
  t.feats = feats;
  t.N = N;
  t.row_bytes = row_bytes;
  t.B = B;
  t.node_cap = node_cap;
  t.n_b = n_b;
  t.packed_ptr_host = packed_ptr_host;
  t.packed_ids = packed_ids;
  t.pinfo = pk.pinfo;
  t.local = pk.local;
  t.loc = loc;
  t.packed = packed;
  t.unc_ids = pk.pw.unc_ids;
  t.unc_off = pk.pw.unc_off;
  t.pairdest = pk.pw.pairdest;
  t.n_unc = sizes->unique_packed;
  t.rows = rows;
  t.err = pk.err;
  int ev_loc = -1, ev_gather = -1;
  if ((rc = pack_fused_tail(t, rows_async, stream, rows_stream, &tm, &ev_loc, &ev_gather)))
    return rc;
  if ((rc = check_err(pk.err, stream))) return rc;
  if (timing) {
    sample_times(tm, mk, timing);
    timing->loc_ms = tm.ms(mk.r1, ev_loc);
    timing->gather_ms = tm.ms(ev_loc, ev_gather);
    timing->total_ms = tm.ms(mk.start, ev_gather);
  }
  return DG_OK;
}
