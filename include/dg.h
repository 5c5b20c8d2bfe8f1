/*
 * dg.h — C ABI of libdg: the group-sampling -> batched-packing -> batch-assembly
 * path of offline-sampling GNN training (DiskGNN, arXiv 2405.05231), on one
 * AMD Instinct MI355X (gfx950).
 *
 * The method (paper §3 "Offline Sampling", §4, §5.2): sample many mini-batches
 * before any model computation, collect the node features each of them will
 * read, and lay those features out in advance.  Three calls cover the path:
 *
 *   dg_sample_group    node-wise fan-out neighbour sampling (§2, Fig. 1) for a
 *                      group of B mini-batches at once.
 *   dg_pack_group      batched feature packing (§5.2, Fig. 6b): deduplicate the
 *                      group's node IDs, drop the nodes held in the feature cache
 *                      (§3 "cache configuration", §4 four-level store), and copy
 *                      each remaining feature row once from the feature table into
 *                      the packed chunk of every mini-batch that needs it; also
 *                      build the per-batch address tables (§6 "interpreted address
 *                      tables").
 *   dg_assemble_batch  feature assembling (§4, Fig. 3): merge cache rows and packed
 *                      rows into one mini-batch's input tensor, in sampled order.
 *
 * Everything lives in device memory (HBM): the disk tiers of the paper are not
 * part of this library.
 *
 * ------------------------------------------------------------------------------
 * Conventions shared by every entry point
 * ------------------------------------------------------------------------------
 *  - Pointers are DEVICE pointers unless the comment says [host].
 *  - Node IDs are int32 in [0, N) (N < 2^31); CSR edge offsets are int64.
 *  - The caller owns every buffer.  The library never allocates device memory:
 *    scratch space is the caller's workspace `ws`, sized by the matching
 *    *_workspace_bytes() query and aligned to 256 bytes (dg_pack_group_noalloc
 *    alone uses a fixed scratch array inside the library instead).  Workspace contents on
 *    entry are irrelevant and on return unspecified, except where the flags
 *    DG_SAMPLE_ENTRY_CLEAR / DG_SAMPLE_EXIT_CLEAR say otherwise.  The only resources
 *    the library takes for itself are a 4 KB page-locked host buffer per calling
 *    thread (for reading counts back) and, per calling thread and device, a few
 *    timing events and a second stream (default priority) on which
 *    dg_pack_group runs part of its work; all are held until the process ends.
 *  - Work is enqueued on the caller's stream `stream` (NULL = the default
 *    stream).  dg_sample_group and dg_pack_group return only when their work has
 *    completed (their output sizes are data-dependent and are reported in
 *    `*sizes`), except for a row copy that dg_pack_group is told to leave on a
 *    second stream (DG_PACK_ROWS_STREAM); dg_assemble_batch is asynchronous.
 *  - Return value: a dg_status.  On a non-OK return dg_last_error() gives a
 *    message (per calling thread).  No exception or abort crosses the ABI.
 *    On DG_ECAPACITY the call stops before writing past any output buffer;
 *    outputs are then unspecified and `*sizes` holds the sizes needed.
 *  - Calls that share a workspace must not overlap in time; calls with distinct
 *    workspaces may run concurrently on different streams.
 *
 * ------------------------------------------------------------------------------
 * Sampling rule (§2 "Graph sampling for GNN training", Fig. 1)
 * ------------------------------------------------------------------------------
 * For each mini-batch b independently, with seeds s_0..s_{S-1} (distinct) and
 * fan-outs f_1..f_K (fanouts[k-1] is hop k):
 *   hop 0 frontier = the seeds, in the given order;
 *   at hop k every node of the hop-(k-1) frontier, in frontier order, draws
 *   min(deg, f_k) distinct neighbour positions of its CSR row (all of them when
 *   f_k < 0 or deg <= f_k), ordered by ascending position; each draw is a
 *   sampled edge (frontier node -> neighbour);
 *   the hop-k frontier = the sampled neighbours not yet in the mini-batch,
 *   deduplicated and sorted by ascending node ID.  Only these newly reached
 *   nodes sample at hop k+1 (in Fig. 1 the seed does not sample again at the
 *   second step).
 * Node list of b:   nodes_b = seeds || hop-1 frontier || ... || hop-K frontier.
 * Edge list of b:   hop by hop; within a hop by frontier position, then by
 *                   ascending CSR position.  Endpoints are local indices into
 *                   nodes_b.
 *
 * Subset drawn when deg d > f (the paper leaves the sampler's randomness to
 * the external framework; this library fixes one, uniform without replacement):
 *   mix64(z): z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9;
 *             z = (z ^ (z >> 27)) * 0x94D049BB133111EB;  return z ^ (z >> 31)
 *             (the SplitMix64 output function; all arithmetic mod 2^64)
 *   gamma   = 0x9E3779B97F4A7C15
 *   key     = mix64( mix64(rng_seed + gamma * (g + 1)) ^ ((uint64)k << 32 | v) )
 *             with g = batch_base + b (the global mini-batch number, as uint64),
 *             k = hop number 1..K, v = the frontier node's ID
 *   h_i     = mix64(key + gamma * (i + 1))      (i-th SplitMix64 output from key)
 *   below(h, m) = floor(h * m / 2^64)           (high word of the 128-bit product)
 *   Floyd's subset (Bentley & Floyd, CACM 30(9), 1987): for i = 0..f-1, with
 *   j = d - f + i, t = below(h_i, j + 1); add t to the subset unless it is
 *   already there, in which case add j.  Positions are then sorted ascending.
 *
 * ------------------------------------------------------------------------------
 * Packing layout (§5.2 "Batched packing", Fig. 6b; §4 "Packed feature chunk")
 * ------------------------------------------------------------------------------
 *   U      = ascending set of all node IDs of the group (its union).
 *   P_b    = ascending IDs of nodes_b whose cache_slot is -1 (not cached): the
 *            packed chunk of b holds exactly the features of P_b, in this order
 *            (batched packing appends features partition by partition in
 *            consecutive-ID order, so each chunk comes out ascending).
 *   packed_ptr[b] = sum_{c<b} |P_c|;  packed row packed_ptr[b]+r = X[P_b[r]].
 *   loc_b[j] = -(cache_slot[u]+1) if u = nodes_b[j] is cached,
 *              else the rank r of u in P_b.
 *   Assembly:  Y_b[j] = cache[-loc_b[j]-1] if loc_b[j] < 0, else packed_b[loc_b[j]],
 *              which equals X[nodes_b[j]] whenever cache row s holds X of the
 *              node whose cache_slot is s.
 * Feature rows are opaque bytes (fp32, fp16, anything): they are copied, never
 * converted.  Rows move as 16-byte vectors when row_bytes and the row base
 * pointers are multiples of 16, and by narrower words otherwise.
 */
#ifndef DG_H
#define DG_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DG_MAX_BATCHES 64 /* a group holds at most 64 mini-batches (one bit each) */

/* dg_sample_group / dg_sample_bounds flags */
#define DG_SAMPLE_LAYERED 1u /* every node of the mini-batch so far samples at each hop
                                (layer-wise blocks as DGL builds them), instead of only
                                the nodes new at the previous hop */
#define DG_SAMPLE_DIRECT 2u  /* relabel sampled neighbours through a direct [N][B]
                                int32 table of local indices (4*N*B workspace bytes)
                                instead of a hash table sized for the group; same
                                results, fewer device-wide atomics */
/* The two flags below let a loop that samples and packs group after group skip
 * clearing two N-word masks per group (2 x 8*N bytes of writes).  Outputs are
 * the same with or without them. */
#define DG_SAMPLE_EXIT_CLEAR 4u   /* on DG_OK, leave the workspace's sampling state
                                     clear (costs a few writes of the last hop) */
#define DG_SAMPLE_ENTRY_CLEAR 8u  /* the caller asserts that `membership` (required)
                                     is all-zero and that the workspace was last used
                                     by a call with DG_SAMPLE_EXIT_CLEAR that returned
                                     DG_OK for the same num_nodes; the call then does
                                     not clear them.  If the assertion is false the
                                     outputs are unspecified (the call still never
                                     accesses memory outside the given buffers). */

/* dg_pack_group flags */
#define DG_PACK_CLEAR_MEMBERSHIP 1u /* on DG_OK, `membership` (required) is left
                                       all-zero: the call clears each word as it
                                       reads it (with member_lines it reads only
                                       the words of marked lines, so the others
                                       must be zero already) */
#define DG_PACK_ROWS_STREAM 2u      /* enqueue the row copy on `rows_stream`, behind the
                                       tables, and return without waiting for it */
#define DG_PACK_LOC_PENDING 4u      /* `loc` already holds what dg_sample_group wrote
                                       into it for these lists and this cache_slot (see
                                       DG_LOC_PENDING): the call completes only the
                                       pending entries and keeps the others */

/* Address-table entry that dg_sample_group leaves for dg_pack_group to fill in
 * (a node that is not cached: its rank in the packed chunk is known only once
 * the whole group is sampled). */
#define DG_LOC_PENDING 0x7fffffff

typedef enum dg_status {
  DG_OK = 0,
  DG_EINVAL = -1,     /* bad argument, or bad input data found by a device check */
  DG_ECAPACITY = -2,  /* an output buffer is too small; see *sizes */
  DG_EHIP = -3,       /* the HIP runtime returned an error */
  DG_EWORKSPACE = -4  /* workspace missing, misaligned or smaller than required */
} dg_status;

/* CSR graph: the neighbours of node v are indices[offsets[v] .. offsets[v+1]).
 * offsets: [N+1] int64, offsets[0] = 0, non-decreasing, offsets[N] = num_edges.
 * indices: [num_edges] int32 node IDs.  Both device pointers. */
typedef struct dg_csr {
  int64_t num_nodes;
  int64_t num_edges;
  const int64_t *offsets;
  const int32_t *indices;
} dg_csr;

/* [host] Sizes reported by dg_sample_group / dg_pack_group.  Fields a call does
 * not compute are set to -1.  exact = 0 means a capacity stop ended the call
 * early and the sampling figures are lower bounds (use dg_sample_bounds()). */
typedef struct dg_sizes {
  int64_t max_batch_nodes; /* max_b n_b: the node_cap needed                */
  int64_t max_batch_edges; /* max_b e_b: the edge_cap needed                */
  int64_t total_nodes;     /* sum_b n_b (= number of (node, batch) pairs)    */
  int64_t total_edges;     /* sum_b e_b                                     */
  int64_t packed_rows;     /* sum_b |P_b|: the packed_cap needed            */
  int64_t unique_nodes;    /* |U|: the unique_cap needed                    */
  int64_t unique_packed;   /* |U minus cached|: feature rows read by packing */
  int32_t exact;
} dg_sizes;

/* [host] Optional per-phase device times in milliseconds, measured with HIP
 * events on the call's stream when a non-NULL pointer is passed.  Phases a call
 * does not run are set to 0. */
typedef struct dg_timing {
  float sample_ms;  /* dg_sample_group: frontier degree pass + draw + mark      */
  float dedup_ms;   /* dg_sample_group: per-hop new-node compaction            */
  float relabel_ms; /* dg_sample_group: global -> local neighbour IDs          */
  float mark_ms;    /* dg_pack_group:   group membership bitmask               */
  float order_ms;   /* dg_pack_group:   unique set, P_b order, packed_ptr      */
  float loc_ms;     /* dg_pack_group:   address tables                         */
  float gather_ms;  /* dg_pack_group:   fan-out row gather (the copy itself)   */
  float total_ms;   /* whole call, first to last enqueued kernel               */
} dg_timing;

/* Library version string (static storage). */
const char *dg_version(void);

/* Message for the last non-OK status returned on the calling thread
 * (thread-local storage; valid until the thread's next dg_* call). */
const char *dg_last_error(void);

/* [host only, no device work] Upper bounds on n_b and e_b for any graph with
 * `num_nodes` nodes and `num_edges` edges and the sampling mode in `flags`.
 * Without DG_SAMPLE_LAYERED: hop k adds at most min(f_k * F_{k-1}, E) edges and
 * as many nodes, where F_0 = S and F_k = the hop's edge bound (only new nodes
 * sample next); with it, F_k = the node bound so far (every node samples).  A
 * negative fan-out counts as E edges; node bounds are capped at N.  For the
 * default mode this gives n_b <= min(N, S*(1 + f1 + f1*f2 + ...)).  Capacities
 * this large never trigger DG_ECAPACITY.  `flags` may be the whole flags word
 * of the sampling call: only DG_SAMPLE_LAYERED changes the bounds.  Returns
 * DG_EINVAL on a null pointer, S < 1, K < 0, num_nodes < 1 or unknown flags. */
int dg_sample_bounds(int64_t num_nodes, int64_t num_edges, int32_t S,
                     const int32_t *fanouts /*[host] K*/, int32_t K, uint32_t flags,
                     int64_t *node_cap /*[host] out*/, int64_t *edge_cap /*[host] out*/);

/* Workspace bytes dg_sample_group needs for N nodes, B batches, the given
 * per-batch capacities and the same flags (DG_SAMPLE_DIRECT adds 4*N*B bytes).
 * Returns 0 for arguments dg_sample_group would reject. */
size_t dg_sample_workspace_bytes(int64_t num_nodes, int32_t B, int64_t node_cap,
                                 int64_t edge_cap, uint32_t flags);

/* Bytes of a member-lines map for N nodes: one byte per 8 consecutive nodes,
 * rounded up to whole blocks of 4096 nodes (512 bytes each). */
size_t dg_member_lines_bytes(int64_t num_nodes);

/* Group sampling (§2 Fig. 1; §3: many mini-batches are sampled before any
 * computation).  Rule and randomness: see the top of this file.
 *   g          CSR graph [host struct, device arrays].
 *   seeds      [B*S] int32; batch b's seeds are seeds[b*S .. b*S+S), distinct
 *              within a batch, each in [0, N).  Batches may share seeds.
 *   B          1..64 mini-batches;  S >= 1 seeds per batch.
 *   batch_base global number of batch 0 (the RNG key uses batch_base + b, so a
 *              group split into several calls gives the same result).
 *   fanouts    [host] K fan-outs, hop 1 first; f < 0 means "all neighbours",
 *              f = 0 samples nothing at that hop.  K >= 0.
 *   rng_seed   sampler seed.
 *   flags      0, or an OR of: DG_SAMPLE_LAYERED: at every hop all nodes of the
 *              mini-batch so far sample (in list order), not only the previous
 *              hop's new nodes; the node list then nests as DGL's layer-wise
 *              blocks do (the first hop_ptr[k] nodes are the destinations of
 *              hop k+1).  DG_SAMPLE_DIRECT: the relabelling table is a direct
 *              [N][B] array (outputs are identical either way).
 *              DG_SAMPLE_EXIT_CLEAR, DG_SAMPLE_ENTRY_CLEAR: see their definitions.
 *              A loop passes EXIT_CLEAR on every call and ENTRY_CLEAR from its
 *              second call on, after a dg_pack_group with
 *              DG_PACK_CLEAR_MEMBERSHIP has cleared the membership words; after
 *              any non-OK return it starts again without ENTRY_CLEAR.
 * Outputs (row b of each starts at b*cap):
 *   nodes      [B*node_cap] int32: nodes_b in the order above.
 *   hop_ptr    [host] [B*(K+2)] int64: hop_ptr[b*(K+2)+h] = start of hop h in
 *              nodes_b (h = 0 is the seeds), hop_ptr[b*(K+2)+K+1] = n_b.
 *   edge_src, edge_dst  [B*edge_cap] int32: sampled edge (frontier node ->
 *              sampled neighbour), both as local indices into nodes_b.
 *   edge_ptr   [host] [B*(K+1)] int64: edge_ptr[b*(K+1)+k] = start of hop-(k+1)
 *              edges, edge_ptr[b*(K+1)+K] = e_b.
 *   membership optional [N] uint64 output (NULL = kept in the workspace): on
 *              return bit b of membership[u] is set iff u is in nodes_b.  It can
 *              be handed to dg_pack_group, which then skips building it.
 *   member_lines  optional [dg_member_lines_bytes(N)] uint8 output: byte i is
 *              non-zero iff one of nodes 8i .. 8i+7 is in some list (bytes past
 *              the last node are 0).  Handed to dg_pack_group with the
 *              membership words, it lets packing read only the words of marked
 *              lines.  The last hop's compaction writes it as it reads every
 *              word; when that hop reads only part of the words (small hops),
 *              a pass over the membership words writes it instead.
 *   cache_slot, loc  optional, both or neither: the address tables of §6 for
 *              the cached nodes, written as the lists are built.  cache_slot
 *              [N] int32 as dg_pack_group takes it (-1 = not cached); loc
 *              [B*node_cap] int32, laid out as nodes: for each entry j of
 *              nodes_b, loc[b*node_cap+j] = -(cache_slot[u]+1) if its node u
 *              is cached, else DG_LOC_PENDING.  dg_pack_group, given the same
 *              lists (node_stride = node_cap), the same cache_slot, this loc and
 *              DG_PACK_LOC_PENDING, completes the pending entries, so that no
 *              cache slot is looked up per entry there.  A cache_slot value
 *              below -1 is reported (DG_EINVAL).
 *   sizes      [host] filled on DG_OK and DG_ECAPACITY.
 *   timing     [host] optional (NULL = not measured).
 * node_cap must be below 2^27.
 * Errors: DG_EINVAL for null pointers, B outside 1..64, S < 1, K < 0, caps < S,
 * unknown flags or DG_SAMPLE_ENTRY_CLEAR without membership, and for bad data
 * found on the device: a seed outside [0,N), a seed repeated in
 * a batch, a CSR row with offsets outside [0,E] or decreasing, a neighbour ID
 * outside [0,N).  Bad data never causes an access outside the given arrays. */
int dg_sample_group(const dg_csr *g, const int32_t *seeds, int32_t B, int32_t S,
                    int64_t batch_base, const int32_t *fanouts, int32_t K,
                    uint64_t rng_seed, uint32_t flags, int64_t node_cap, int32_t *nodes,
                    int64_t *hop_ptr, int64_t edge_cap, int32_t *edge_src,
                    int32_t *edge_dst, int64_t *edge_ptr, uint64_t *membership,
                    uint8_t *member_lines, const int32_t *cache_slot, int32_t *loc,
                    void *ws, size_t ws_bytes, hipStream_t stream, dg_sizes *sizes,
                    dg_timing *timing);

/* Workspace bytes dg_pack_group needs for N nodes, B batches whose node lists
 * hold `total_nodes` entries in all. */
size_t dg_pack_workspace_bytes(int64_t num_nodes, int32_t B, int64_t total_nodes);

/* Batched packing (§5.2 Fig. 6b) + address tables (§6).  Layout: see the top of
 * this file.
 *   feats       [N*row_bytes] feature table X, row v at feats + v*row_bytes.
 *   N, row_bytes  row_bytes >= 1.
 *   cache_slot  [N] int32: row of node v in the cache table, or -1 if not cached.
 *   B           1..64;  nodes [B*node_stride] int32, batch b's list at
 *               nodes + b*node_stride, distinct within a batch (any order: the
 *               lists may come from any sampler, §3 "Generality").
 *   node_count  [host] [B] int64: n_b (0 <= n_b <= node_stride).
 * Outputs:
 *   packed      [packed_cap*row_bytes] bytes: the packed chunks, batch-major;
 *               NULL = build the tables below without copying any row.
 *   packed_ids  [packed_cap] int32: node ID of each packed row (P_0 || P_1 ...).
 *   packed_ptr  [B+1] int64 (device) and packed_ptr_host [host] [B+1] int64:
 *               chunk b is rows packed_ptr[b] .. packed_ptr[b+1).
 *   loc         [B*node_stride] int32: address table, loc_b at loc + b*node_stride.
 *   group_unique  [unique_cap] int32 or NULL: U ascending.
 *   membership  optional [N] uint64 input (NULL = built here from the lists):
 *               bit b of membership[u] set iff u is in batch b's list, as
 *               dg_sample_group returns it; bits of batches >= B are ignored.
 *               Read only, unless flags holds DG_PACK_CLEAR_MEMBERSHIP.
 *   member_lines  optional (with membership) [dg_member_lines_bytes(N)] uint8, as
 *               dg_sample_group writes it: words of lines whose byte is 0 are
 *               not read.  A member in an unmarked line is missed, which the
 *               pair-count check reports (DG_EINVAL).
 *   cache_nodes, cache_rows, cache_table  optional cache fill (NULL cache_table =
 *               none): the caches are filled by batched packing as special
 *               mini-batches (§5.2), so the row copy also reads the row of each
 *               cache_nodes[s] (s < cache_rows) once and writes it to row s of
 *               cache_table [cache_rows*row_bytes], in the same gather launch as
 *               the packed chunks.  A slot holding -1 is left as it is; another
 *               ID outside [0, N) is reported (DG_EINVAL).  Needs packed, and
 *               cannot be combined with DG_PACK_ROWS_STREAM.
 *   flags       0, or an OR of DG_PACK_CLEAR_MEMBERSHIP, DG_PACK_ROWS_STREAM and
 *               DG_PACK_LOC_PENDING.  With DG_PACK_LOC_PENDING, loc must hold
 *               what dg_sample_group wrote for these lists and this cache_slot:
 *               entries that are not DG_LOC_PENDING are kept as they are (a
 *               cached node's entry), and a pending entry whose node turns out
 *               to be cached, or to lack its membership bit, is reported
 *               (DG_EINVAL).
 *   rows_stream used only with DG_PACK_ROWS_STREAM (and packed != NULL): the row
 *               copy, which reads feats and the workspace and writes packed, is
 *               enqueued there after an event that follows the tables on
 *               `stream`, and the call returns when the tables are done.  Work
 *               the caller queues on rows_stream after the call sees `packed`
 *               complete.  Until the copy has run, the workspace must not be
 *               reused and feats and packed must not be written.  This lets a
 *               pipeline run the bandwidth-bound copy beside the next group's
 *               sampling.
 *               The call checks that the bit of every non-cached list entry is
 *               set and that the mask holds as many (node, batch) pairs as the
 *               lists have entries (DG_EINVAL otherwise); a mask that passes these
 *               checks and still differs from the lists gives unspecified packing
 *               outputs, never an access outside the given buffers.
 *   sizes, timing as for dg_sample_group.  Without timing the address tables
 *               are built on the library's second stream while the row copy
 *               runs on `stream` (both done before the call returns); with
 *               timing the phases run one after the other.  timing cannot be
 *               combined with DG_PACK_ROWS_STREAM.
 * Errors: DG_EINVAL for null pointers, B outside 1..64, row_bytes < 1, n_b out of
 * range, unknown flags (or DG_PACK_CLEAR_MEMBERSHIP or member_lines without
 * membership), and on
 * the device a node ID outside [0,N), a node repeated within a batch, or
 * cache_slot[v] < -1.  DG_ECAPACITY when packed_cap < sum|P_b| or
 * (group_unique != NULL and) unique_cap < |U|. */
int dg_pack_group(const void *feats, int64_t N, int64_t row_bytes,
                  const int32_t *cache_slot, int32_t B, const int32_t *nodes,
                  int64_t node_stride, const int64_t *node_count, int64_t packed_cap,
                  void *packed, int32_t *packed_ids, int64_t *packed_ptr,
                  int64_t *packed_ptr_host, int32_t *loc, int32_t *group_unique,
                  int64_t unique_cap, uint64_t *membership, const uint8_t *member_lines,
                  const int32_t *cache_nodes, int64_t cache_rows, void *cache_table,
                  uint32_t flags, void *ws, size_t ws_bytes, hipStream_t stream,
                  hipStream_t rows_stream, dg_sizes *sizes, dg_timing *timing);

/* Bytes of the packing workspace dg_sample_pack_group needs for N nodes, B
 * batches and per-batch capacity node_cap (room for B*node_cap list entries).
 * Returns 0 for B outside 1..64, N < 1 or node_cap < 1. */
size_t dg_sample_pack_workspace_bytes(int64_t num_nodes, int32_t B, int64_t node_cap);

/* Group sampling and batched packing in one call (§3 offline sampling, §5.2
 * batched packing, §6 address tables).  The outputs are those of
 *   dg_sample_group(g, ..., flags, node_cap, nodes, hop_ptr, edge_cap, edge_src,
 *                   edge_dst, edge_ptr, membership, NULL, cache_slot, loc, ws, ...)
 * followed by
 *   dg_pack_group(feats, N, row_bytes, cache_slot, B, nodes, node_cap, n_b,
 *                 packed_cap, packed, packed_ids, packed_ptr, packed_ptr_host, loc,
 *                 group_unique, unique_cap, membership, <member lines>, NULL, 0,
 *                 NULL, DG_PACK_CLEAR_MEMBERSHIP | DG_PACK_LOC_PENDING | pack_flags,
 *                 ...)
 * with n_b = hop_ptr[b*(K+2)+K+1]: the same nodes, edges, address tables, U,
 * P_b, packed_ptr and packed rows, and `membership` (or the workspace's copy)
 * left all-zero on DG_OK.
 * With DG_SAMPLE_DIRECT and a last hop that samples, the two do not run one
 * after the other: the last hop's compaction, which reads every membership
 * word once the group is complete, also produces packing's sets (U, U_nc,
 * each P_b, every pair's packed row) from that same read, and the address
 * tables of non-cached entries follow from one read of the direct table per
 * older pair.  Otherwise (hash relabelling, a last hop with fan-out 0 or an
 * empty frontier, K = 0) packing's own passes run after sampling.
 *   Arguments as for dg_sample_group and dg_pack_group; cache_slot, loc and
 *   feats are required, and loc is laid out as nodes (node_stride = node_cap).
 *   pack_flags  0 or DG_PACK_ROWS_STREAM (rows_stream as for dg_pack_group: the
 *               row copy is queued there and not waited for; until it has run,
 *               pack_ws must not be reused and feats and packed must not be
 *               written).
 *   ws, ws_bytes        sampling's workspace (dg_sample_workspace_bytes).
 *   pack_ws, pack_ws_bytes  packing's (dg_sample_pack_workspace_bytes), 256-aligned.
 *   sizes       [host] every field (sampling's and packing's).
 *   timing      optional: sampling's phases, then loc_ms (address tables after
 *               the fused pass) and gather_ms; mark_ms and order_ms are 0 when
 *               the passes were fused (their work is inside dedup_ms).
 * Errors: those of the two calls; DG_EWORKSPACE for a missing, small or
 * misaligned pack_ws.  After a non-OK return the membership words and the
 * workspaces are in an unspecified state (start again without
 * DG_SAMPLE_ENTRY_CLEAR). */
int dg_sample_pack_group(const dg_csr *g, const int32_t *seeds, int32_t B, int32_t S,
                         int64_t batch_base, const int32_t *fanouts, int32_t K,
                         uint64_t rng_seed, uint32_t flags, int64_t node_cap, int32_t *nodes,
                         int64_t *hop_ptr, int64_t edge_cap, int32_t *edge_src,
                         int32_t *edge_dst, int64_t *edge_ptr, uint64_t *membership,
                         const int32_t *cache_slot, int32_t *loc, const void *feats,
                         int64_t row_bytes, int64_t packed_cap, void *packed,
                         int32_t *packed_ids, int64_t *packed_ptr, int64_t *packed_ptr_host,
                         int32_t *group_unique, int64_t unique_cap, uint32_t pack_flags,
                         void *ws, size_t ws_bytes, void *pack_ws, size_t pack_ws_bytes,
                         hipStream_t stream, hipStream_t rows_stream, dg_sizes *sizes,
                         dg_timing *timing);

/* Bytes of the fixed scratch of dg_pack_group_noalloc (256 MiB). */
size_t dg_pack_noalloc_scratch_bytes(void);

/* dg_pack_group for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments, outputs and errors, except that the call allocates nothing.
 *  - Its scratch is a fixed array inside the library, one per GPU, of
 *    dg_pack_noalloc_scratch_bytes() bytes; each GPU the library runs on holds
 *    it until the process ends.  Calls whose sizes need more
 *    (dg_pack_workspace_bytes(N, B, sum of n_b) above that) return
 *    DG_EWORKSPACE before any work is enqueued.
 *  - Every call on a GPU shares that GPU's scratch, which keeps the last
 *    call's contents; each call clears what it needs cleared.  Calls that
 *    overlap in time on one GPU race and give unspecified outputs: the caller
 *    must serialise them (across host threads and streams).
 *  - All work runs on `stream`: no second stream, so DG_PACK_ROWS_STREAM is
 *    rejected (DG_EINVAL) and no timing is taken.  Counts are read back
 *    straight into host memory, with no page-locked buffer of the library's.
 *  - No hipMalloc, hipHostMalloc, hipFree, stream or event creation. */
int dg_pack_group_noalloc(const void *feats, int64_t N, int64_t row_bytes,
                          const int32_t *cache_slot, int32_t B, const int32_t *nodes,
                          int64_t node_stride, const int64_t *node_count, int64_t packed_cap,
                          void *packed, int32_t *packed_ids, int64_t *packed_ptr,
                          int64_t *packed_ptr_host, int32_t *loc, int32_t *group_unique,
                          int64_t unique_cap, uint64_t *membership,
                          const uint8_t *member_lines, const int32_t *cache_nodes,
                          int64_t cache_rows, void *cache_table, uint32_t flags,
                          hipStream_t stream, dg_sizes *sizes);

/* Feature assembling for one mini-batch (§4 Fig. 3, second step; addresses come
 * from the precomputed table of §6, so no lookup structure is consulted):
 *   out[j] = cache[-loc_b[j]-1] if loc_b[j] < 0, else packed_b[loc_b[j]],
 *   for j in [0, n_b); each row is row_bytes bytes.
 *   cache      [cache_rows*row_bytes] the cache table (may be NULL if cache_rows=0).
 *   packed_b   [packed_rows_b*row_bytes] = packed + packed_ptr[b]*row_bytes.
 *   loc_b      [n_b] int32;  out [n_b*row_bytes].
 *   status     optional device int32: on an entry of loc_b outside
 *              [-cache_rows, packed_rows_b) the kernel writes a zero row and ORs
 *              1 (bit 0) into *status.  It reads no table row for such an entry
 *              (only the out row it then overwrites), so no access falls outside
 *              the given buffers.
 * Asynchronous on `stream`.  Returns DG_EINVAL for null pointers (other than
 * cache with cache_rows = 0 and status), n_b < 0, row_bytes < 1, or buffers that
 * overlap; n_b = 0 is a no-op. */
int dg_assemble_batch(const void *cache, int64_t cache_rows, const void *packed_b,
                      int64_t packed_rows_b, const int32_t *loc_b, int64_t n_b,
                      int64_t row_bytes, void *out, int32_t *status,
                      hipStream_t stream);

/* dg_assemble_batch for batches 0..B-1 of one packing result, in batch order on
 * `stream`, issued by one call.  Up to eight consecutive batches whose output
 * buffers are distinct and apart (and whose rows move as 16-byte vectors) share
 * one kernel launch; the outputs are those of the per-batch calls in batch
 * order either way.
 *   packed, packed_ptr_host [host] [B+1]  the packed chunks and their bounds as
 *              dg_pack_group returned them (packed may be NULL if every chunk is
 *              empty).
 *   loc        [B*loc_stride] address tables; node_count [host] [B] the n_b.
 *   outs       [host] [n_outs] output buffers; batch b goes to outs[b % n_outs],
 *              each buffer at least max_b n_b * row_bytes bytes.  Batches that
 *              share a buffer overwrite it in batch order.
 * Asynchronous on `stream`.  DG_EINVAL, before anything is enqueued, for
 * B < 0, n_outs < 1, row_bytes < 1, a null outs/packed_ptr_host/node_count, or
 * any batch with n_b > loc_stride or chunk bounds that decrease.  Each batch is
 * then checked as dg_assemble_batch checks it; the call stops at the first
 * batch that fails (batches before it are already enqueued) and returns that
 * status. */
int dg_assemble_batches(const void *cache, int64_t cache_rows, const void *packed,
                        const int64_t *packed_ptr_host, const int32_t *loc,
                        int64_t loc_stride, const int64_t *node_count, int32_t B,
                        int64_t row_bytes, void *const *outs, int32_t n_outs,
                        int32_t *status, hipStream_t stream);

/* Workspace bytes dg_cache_by_frequency needs for N nodes. */
size_t dg_cache_workspace_bytes(int64_t num_nodes);

/* Cache configuration by access frequency (§4 "Four-level hierarchical feature
 * store": a counter per node over the graph samples; §3 "Cache configuration":
 * caching the most frequently accessed features minimises the features left to
 * fetch from slower storage).  The access count of node u is the number of the
 * group's mini-batches that require it: popcount(membership[u] & batch bits),
 * with membership as dg_sample_group returns it.  Nodes are ranked by count,
 * descending, ties by ascending ID; the first min(cache_rows, #accessed)
 * nodes are cached.
 *   cache_slot   [N] int32 out: rank of u if cached, else -1.
 *   cache_nodes  [cache_rows] int32 out: cached node of each slot; -1 for
 *                slots left empty (fewer accessed nodes than cache_rows).
 *   cached       [host] out: number of cached nodes.
 * Returns after completion.  DG_EINVAL for null pointers, B outside 1..64,
 * cache_rows outside [0, N]; DG_EWORKSPACE for a small workspace. */
int dg_cache_by_frequency(const uint64_t *membership, int64_t N, int32_t B, int64_t cache_rows,
                          int32_t *cache_slot, int32_t *cache_nodes, int64_t *cached, void *ws,
                          size_t ws_bytes, hipStream_t stream);

/* Row gather: out[i] = feats[ids[i]] for i in [0, n) (rows of row_bytes
 * bytes).  Fills the cache table from dg_cache_by_frequency's cache_nodes (the
 * paper fills its caches by batched packing, treating each cache as one more
 * mini-batch, §5.2), and, called once per mini-batch over that batch's
 * packed_ids, performs the individual packing of §5.2 (Fig. 6a) that batched
 * packing replaces.  An id outside [0, N) writes a zero row and ORs 1 (bit 0)
 * into the optional device int32 *status; it reads no row of feats (only the
 * out row it then overwrites).  Asynchronous on `stream`.
 * DG_EINVAL for bad sizes, null pointers or an output overlapping an input. */
int dg_gather_rows(const void *feats, int64_t N, int64_t row_bytes, const int32_t *ids,
                   int64_t n, void *out, int32_t *status, hipStream_t stream);

/* Workspace bytes dg_minhash_order needs for m disk-cache entries. */
size_t dg_minhash_workspace_bytes(int64_t m);

/* Disk-cache node reordering by MinHash (§5.1 "Node reordering for disk
 * cache", Alg. 1, after HashOrder): features that the same graph samples
 * require are placed next to each other.
 *   membership  [N] uint64: bit i of membership[v] set iff graph sample
 *               (mini-batch) i requires v, i < B (as dg_sample_group returns).
 *   entries     [m] int32: the disk-cache nodes V_d, in their current order.
 *   perms       [k*B] int32 (device): hash function j maps sample i to
 *               perms[j*B + i], a permutation of 0..B-1 (the random
 *               permutations are drawn by the caller).
 *   S(v) = min over every j and every sample i requiring v of perms[j*B + i]
 *   (one running minimum across the k functions, as the algorithm writes it);
 *   S(v) = infinity when no sample requires v.
 *   order       [m] int32 out: V_d stably sorted by S (ties keep entry order,
 *               entries required by no sample last).
 *   signature   [m] int32 out, optional: S of each entry (-1 = infinity).
 * Returns after completion.  DG_EINVAL for null pointers, B outside 1..64,
 * k < 1, an entry outside [0, N) or a hash value outside [0, B). */
int dg_minhash_order(const uint64_t *membership, int64_t N, int32_t B, const int32_t *entries,
                     int64_t m, const int32_t *perms, int32_t k, int32_t *order,
                     int32_t *signature, void *ws, size_t ws_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* DG_H */
