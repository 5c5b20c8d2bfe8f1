/*
 * oracle.c — plain, slow, single-threaded CPU reference for the offline-sampling
 * path (group sampling, batched packing, batch assembly) of DiskGNN
 * (arXiv 2405.05231).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code with
 * the device library: it is written from the paper's definitions, with plain
 * loops, qsort and bsearch, in the paper's order of steps, so that each function
 * can be checked against the text by eye.
 *
 * Pins (tests that tie this code to something other than itself): the paper's
 * worked examples for Fig. 1 (§2/§3), Fig. 3 (§4) and Fig. 6 (§5.2); brute-force
 * set computations on tiny graphs; the breadth-first-search special case; the
 * published SplitMix64 output sequence; chi-square uniformity of the drawn
 * subsets.  The particular subset drawn for a given key follows the written RNG
 * rule (the paper leaves the sampler's randomness open): that choice is
 * "parity unpinned" against any external sampler.
 *
 * All functions return 0 on success and a negative code on error:
 *   -1 bad argument or bad input data, -2 a capacity is too small.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------------------
 * Randomness of the sampler (the paper leaves it to the external sampling
 * framework; the rule here is the library's written one).
 * ------------------------------------------------------------------------- */

/* SplitMix64 output function (Steele, Lea & Flood, OOPSLA 2014). */
uint64_t or_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static const uint64_t OR_GAMMA = 0x9E3779B97F4A7C15ULL;

/* i-th output (i = 0, 1, ...) of a SplitMix64 generator whose state starts at
 * `state`: the state advances by gamma before each output. */
uint64_t or_splitmix_nth(uint64_t state, uint64_t i) {
  return or_mix64(state + OR_GAMMA * (i + 1));
}

/* Key of one frontier node's draw: global batch number g, hop k (1-based),
 * node v. */
uint64_t or_draw_key(uint64_t rng_seed, uint64_t g, int32_t k, int32_t v) {
  uint64_t batch_state = or_mix64(rng_seed + OR_GAMMA * (g + 1));
  return or_mix64(batch_state ^ (((uint64_t)(uint32_t)k << 32) | (uint64_t)(uint32_t)v));
}

/* floor(h * m / 2^64): maps a 64-bit draw onto [0, m). */
uint64_t or_below(uint64_t h, uint64_t m) {
  unsigned __int128 p = (unsigned __int128)h * (unsigned __int128)m;
  return (uint64_t)(p >> 64);
}

static int cmp_i64(const void *a, const void *b) {
  int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  return (x > y) - (x < y);
}
static int cmp_i32(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x > y) - (x < y);
}

/* Floyd's algorithm (Bentley & Floyd, "A sample of brilliance", CACM 1987):
 * a uniform f-subset of {0..d-1}, f <= d.  Step i (0-based) considers
 * j = d - f + i, draws t uniform in {0..j}, and adds t, or j if t was already
 * chosen.  The chosen positions are returned sorted ascending in out[0..f). */
int or_floyd(int64_t d, int32_t f, uint64_t key, int64_t *out) {
  if (f < 0 || d < 0 || (int64_t)f > d) return -1;
  for (int32_t i = 0; i < f; ++i) {
    int64_t j = d - f + i;
    int64_t t = (int64_t)or_below(or_splitmix_nth(key, (uint64_t)i), (uint64_t)(j + 1));
    int seen = 0;
    for (int32_t m = 0; m < i; ++m)
      if (out[m] == t) seen = 1;
    out[i] = seen ? j : t;
  }
  qsort(out, (size_t)f, sizeof(int64_t), cmp_i64);
  return 0;
}

/* ---------------------------------------------------------------------------
 * Group sampling: node-wise fan-out sampling (§2, Fig. 1), run for every
 * mini-batch of the group before any computation (§3 offline sampling).
 * ------------------------------------------------------------------------- */

/* Positions of the neighbours drawn by node v at hop k (1-based):
 * all of 0..d-1 when f < 0 or d <= f, else Floyd's f-subset.  Returns the count. */
static int64_t draw_positions(int64_t d, int32_t f, uint64_t rng_seed, uint64_t g,
                              int32_t k, int32_t v, int64_t *pos) {
  if (f < 0 || d <= (int64_t)f) {
    for (int64_t p = 0; p < d; ++p) pos[p] = p;
    return d;
  }
  or_floyd(d, f, or_draw_key(rng_seed, g, k, v), pos);
  return f;
}

/* layered = 0: only the nodes first reached at hop k sample at hop k+1 (§2,
 * Fig. 1: the seed does not sample again at the second step).
 * layered = 1: every node of the mini-batch so far samples at each hop
 * (layer-wise blocks as DGL builds them). */
int or_sample_group(int64_t N, int64_t E, const int64_t *off, const int32_t *idx,
                    const int32_t *seeds, int32_t B, int32_t S, int64_t batch_base,
                    const int32_t *fanouts, int32_t K, uint64_t rng_seed, int32_t layered,
                    int64_t node_cap, int32_t *nodes, int64_t *hop_ptr,
                    int64_t edge_cap, int32_t *edge_src, int32_t *edge_dst,
                    int64_t *edge_ptr, int64_t *need /* [2]: max n_b, max e_b */) {
  if (N < 1 || B < 1 || S < 1 || K < 0) return -1;
  /* local[u] = index of u in the current batch's node list, or -1 */
  int32_t *local = (int32_t *)malloc((size_t)N * sizeof(int32_t));
  int64_t max_deg = 0;
  for (int64_t v = 0; v < N; ++v) {
    local[v] = -1;
    if (off[v + 1] - off[v] > max_deg) max_deg = off[v + 1] - off[v];
  }
  int64_t *pos = (int64_t *)malloc((size_t)(max_deg + 1) * sizeof(int64_t));
  int64_t cand_cap = 1024, *cand_src = NULL;
  int32_t *cand_nbr = NULL, *fresh = NULL;
  cand_src = (int64_t *)malloc((size_t)cand_cap * sizeof(int64_t));
  cand_nbr = (int32_t *)malloc((size_t)cand_cap * sizeof(int32_t));
  fresh = (int32_t *)malloc((size_t)cand_cap * sizeof(int32_t));
  int rc = 0;
  need[0] = need[1] = 0;
  if (off[0] != 0 || off[N] != E) rc = -1;

  for (int32_t b = 0; b < B && rc == 0; ++b) {
    uint64_t g = (uint64_t)(batch_base + b);
    int32_t *nb = nodes + (int64_t)b * node_cap;
    int64_t *hp = hop_ptr + (int64_t)b * (K + 2);
    int64_t *ep = edge_ptr + (int64_t)b * (K + 1);
    int64_t n = 0, e = 0;

    /* hop 0: the seeds, in the given order */
    for (int32_t i = 0; i < S; ++i) {
      int32_t v = seeds[(int64_t)b * S + i];
      if (v < 0 || v >= N || local[v] >= 0) { rc = -1; break; }
      if (n >= node_cap) { rc = -2; break; }
      nb[n] = v;
      local[v] = (int32_t)n;
      ++n;
    }
    hp[0] = 0;
    hp[1] = n;
    int64_t front_begin = 0, front_end = n;

    for (int32_t k = 1; k <= K && rc == 0; ++k) {
      ep[k - 1] = e;
      int32_t f = fanouts[k - 1];
      int64_t ncand = 0;
      /* every frontier node, in frontier order, draws its neighbours */
      for (int64_t p = front_begin; p < front_end && rc == 0; ++p) {
        int32_t v = nb[p];
        int64_t d = off[v + 1] - off[v];
        int64_t c = draw_positions(d, f, rng_seed, g, k, v, pos);
        for (int64_t q = 0; q < c; ++q) {
          int32_t u = idx[off[v] + pos[q]];
          if (u < 0 || u >= N) { rc = -1; break; }
          if (ncand == cand_cap) {
            cand_cap *= 2;
            cand_src = (int64_t *)realloc(cand_src, (size_t)cand_cap * sizeof(int64_t));
            cand_nbr = (int32_t *)realloc(cand_nbr, (size_t)cand_cap * sizeof(int32_t));
            fresh = (int32_t *)realloc(fresh, (size_t)cand_cap * sizeof(int32_t));
          }
          cand_src[ncand] = p;
          cand_nbr[ncand] = u;
          ++ncand;
        }
      }
      if (rc) break;
      /* the new frontier: sampled neighbours not yet in the batch, ascending */
      int64_t nfresh = 0;
      for (int64_t c = 0; c < ncand; ++c)
        if (local[cand_nbr[c]] < 0) fresh[nfresh++] = cand_nbr[c];
      qsort(fresh, (size_t)nfresh, sizeof(int32_t), cmp_i32);
      int64_t nnew = 0;
      for (int64_t c = 0; c < nfresh; ++c)
        if (c == 0 || fresh[c] != fresh[c - 1]) fresh[nnew++] = fresh[c];
      if (n + nnew > node_cap || e + ncand > edge_cap) {
        rc = -2;
        if (n + nnew > need[0]) need[0] = n + nnew;
        if (e + ncand > need[1]) need[1] = e + ncand;
        break;
      }
      for (int64_t c = 0; c < nnew; ++c) {
        nb[n] = fresh[c];
        local[fresh[c]] = (int32_t)n;
        ++n;
      }
      /* edges with local endpoints */
      int32_t *es = edge_src + (int64_t)b * edge_cap;
      int32_t *ed = edge_dst + (int64_t)b * edge_cap;
      for (int64_t c = 0; c < ncand; ++c) {
        es[e] = (int32_t)cand_src[c];
        ed[e] = local[cand_nbr[c]];
        ++e;
      }
      hp[k + 1] = n;
      front_begin = layered ? 0 : front_end;
      front_end = n;
    }
    if (rc == 0) {
      ep[K] = e;
      if (n > need[0]) need[0] = n;
      if (e > need[1]) need[1] = e;
    }
    /* forget this batch */
    for (int64_t i = 0; i < n; ++i) local[nb[i]] = -1;
  }
  free(local);
  free(pos);
  free(cand_src);
  free(cand_nbr);
  free(fresh);
  return rc;
}

/* ---------------------------------------------------------------------------
 * Batched packing (§5.2, Fig. 6b) and address tables (§6).
 * Written as its closed form: P_b = sorted non-cached nodes of batch b, packed
 * row i = X[packed_ids[i]], U = sorted union, loc from the two.
 * ------------------------------------------------------------------------- */

static int64_t find_i32(const int32_t *sorted, int64_t n, int32_t key) {
  const int32_t *hit = (const int32_t *)bsearch(&key, sorted, (size_t)n, sizeof(int32_t), cmp_i32);
  return hit ? (int64_t)(hit - sorted) : -1;
}

int or_pack_group(int64_t N, int64_t row_bytes, const void *feats, const int32_t *cache_slot,
                  int32_t B, const int32_t *nodes, int64_t node_stride,
                  const int64_t *node_count, int64_t packed_cap, void *packed,
                  int32_t *packed_ids, int64_t *packed_ptr, int32_t *loc,
                  int32_t *group_unique, int64_t unique_cap,
                  int64_t *need /* [3]: packed rows, |U|, |U minus cached| */) {
  if (N < 1 || B < 1 || row_bytes < 1) return -1;
  int64_t total = 0;
  for (int32_t b = 0; b < B; ++b) {
    if (node_count[b] < 0 || node_count[b] > node_stride) return -1;
    total += node_count[b];
  }
  /* input checks: IDs in range, distinct within a batch, cache_slot >= -1 */
  for (int32_t b = 0; b < B; ++b) {
    int64_t nbb = node_count[b];
    int32_t *tmp = (int32_t *)malloc((size_t)(nbb + 1) * sizeof(int32_t));
    memcpy(tmp, nodes + (int64_t)b * node_stride, (size_t)nbb * sizeof(int32_t));
    qsort(tmp, (size_t)nbb, sizeof(int32_t), cmp_i32);
    int bad = 0;
    for (int64_t j = 0; j < nbb; ++j) {
      if (tmp[j] < 0 || tmp[j] >= N || (j > 0 && tmp[j] == tmp[j - 1])) bad = 1;
      else if (cache_slot[tmp[j]] < -1) bad = 1;
    }
    free(tmp);
    if (bad) return -1;
  }

  /* U: sorted union of all node lists */
  int32_t *all = (int32_t *)malloc((size_t)(total + 1) * sizeof(int32_t));
  int64_t t = 0;
  for (int32_t b = 0; b < B; ++b)
    for (int64_t j = 0; j < node_count[b]; ++j) all[t++] = nodes[(int64_t)b * node_stride + j];
  qsort(all, (size_t)total, sizeof(int32_t), cmp_i32);
  int64_t nu = 0, nu_packed = 0;
  for (int64_t i = 0; i < total; ++i)
    if (i == 0 || all[i] != all[i - 1]) {
      all[nu++] = all[i];
      if (cache_slot[all[nu - 1]] < 0) ++nu_packed;
    }

  /* P_b: sorted non-cached nodes of each batch; packed_ptr: running sum */
  int64_t rows = 0;
  for (int32_t b = 0; b < B; ++b)
    for (int64_t j = 0; j < node_count[b]; ++j)
      if (cache_slot[nodes[(int64_t)b * node_stride + j]] < 0) ++rows;
  need[0] = rows;
  need[1] = nu;
  need[2] = nu_packed;
  if (rows > packed_cap || (group_unique && nu > unique_cap)) {
    free(all);
    return -2;
  }
  if (group_unique) memcpy(group_unique, all, (size_t)nu * sizeof(int32_t));
  free(all);

  packed_ptr[0] = 0;
  for (int32_t b = 0; b < B; ++b) {
    const int32_t *nb = nodes + (int64_t)b * node_stride;
    int32_t *pb = packed_ids + packed_ptr[b];
    int64_t cnt = 0;
    for (int64_t j = 0; j < node_count[b]; ++j)
      if (cache_slot[nb[j]] < 0) pb[cnt++] = nb[j];
    qsort(pb, (size_t)cnt, sizeof(int32_t), cmp_i32);
    packed_ptr[b + 1] = packed_ptr[b] + cnt;
    /* address table: cached -> -(slot+1), packed -> rank in P_b */
    for (int64_t j = 0; j < node_count[b]; ++j) {
      int32_t u = nb[j];
      loc[(int64_t)b * node_stride + j] =
          cache_slot[u] >= 0 ? -(cache_slot[u] + 1) : (int32_t)find_i32(pb, cnt, u);
    }
  }
  /* packed row i holds the feature row of node packed_ids[i]
     (packed == NULL: tables only, no row copies) */
  for (int64_t i = 0; packed && i < rows; ++i)
    memcpy((char *)packed + i * row_bytes, (const char *)feats + (int64_t)packed_ids[i] * row_bytes,
           (size_t)row_bytes);
  return 0;
}

/* ---------------------------------------------------------------------------
 * Feature assembling (§4, Fig. 3): each required feature comes from the cache
 * or from the batch's packed chunk, at the address the table gives.
 * ------------------------------------------------------------------------- */
int or_assemble_batch(const void *cache, int64_t cache_rows, const void *packed_b,
                      int64_t packed_rows_b, const int32_t *loc_b, int64_t n_b,
                      int64_t row_bytes, void *out) {
  for (int64_t j = 0; j < n_b; ++j) {
    int32_t l = loc_b[j];
    const char *src;
    if (l < 0) {
      if ((int64_t)(-(int64_t)l - 1) >= cache_rows) return -1;
      src = (const char *)cache + (int64_t)(-(int64_t)l - 1) * row_bytes;
    } else {
      if ((int64_t)l >= packed_rows_b) return -1;
      src = (const char *)packed_b + (int64_t)l * row_bytes;
    }
    memcpy((char *)out + j * row_bytes, src, (size_t)row_bytes);
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * Cache configuration by access frequency (§4: one counter per node, streamed
 * over the graph samples; the most popular features go to the fastest tier).
 * A mini-batch requires each of its nodes once, so a node's count is the
 * number of node lists that hold it.  Ranking: count descending, ties by
 * ascending node ID; only accessed nodes are cached.
 * ------------------------------------------------------------------------- */
static const int64_t *g_rank_count; /* qsort has no context argument */

static int cmp_by_count(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  if (g_rank_count[x] != g_rank_count[y]) return g_rank_count[x] > g_rank_count[y] ? -1 : 1;
  return (x > y) - (x < y);
}

int or_cache_by_frequency(int64_t N, int32_t B, const int32_t *nodes, int64_t node_stride,
                          const int64_t *node_count, int64_t cache_rows, int32_t *cache_slot,
                          int32_t *cache_nodes, int64_t *cached) {
  if (N < 1 || B < 1 || cache_rows < 0 || cache_rows > N) return -1;
  int64_t *count = (int64_t *)calloc((size_t)N, sizeof(int64_t));
  for (int32_t b = 0; b < B; ++b)
    for (int64_t j = 0; j < node_count[b]; ++j) {
      int32_t u = nodes[(int64_t)b * node_stride + j];
      if (u < 0 || u >= N) { free(count); return -1; }
      count[u] += 1;
    }
  int32_t *order = (int32_t *)malloc((size_t)N * sizeof(int32_t));
  for (int64_t v = 0; v < N; ++v) order[v] = (int32_t)v;
  g_rank_count = count;
  qsort(order, (size_t)N, sizeof(int32_t), cmp_by_count);
  int64_t c = 0;
  for (int64_t v = 0; v < N; ++v) cache_slot[v] = -1;
  for (int64_t r = 0; r < cache_rows; ++r) cache_nodes[r] = -1;
  for (int64_t r = 0; r < cache_rows && count[order[r]] > 0; ++r) {
    cache_slot[order[r]] = (int32_t)r;
    cache_nodes[r] = order[r];
    ++c;
  }
  *cached = c;
  free(order);
  free(count);
  return 0;
}

/* ---------------------------------------------------------------------------
 * Disk-cache reordering by MinHash (§5.1, Alg. 1), from its definition: the
 * value of a disk-cache entry v is
 *     S(v) = min { H_j(i) : j a hash function, i a graph sample requiring v },
 * one minimum over all functions and samples together, as the algorithm keeps
 * a single running minimum per node (infinity when no sample requires v);
 * H_j(i) = perms[j*B + i] (permutations drawn by the caller).  The entries are
 * then ordered by S, stably, so ties keep entry order.
 * ------------------------------------------------------------------------- */
typedef struct { int64_t s; int64_t pos; } or_sig;

static int cmp_sig(const void *a, const void *b) {
  const or_sig *x = (const or_sig *)a, *y = (const or_sig *)b;
  if (x->s != y->s) return x->s < y->s ? -1 : 1;
  return (x->pos > y->pos) - (x->pos < y->pos);
}

int or_minhash_order(int64_t N, int32_t B, const int32_t *nodes, int64_t node_stride,
                     const int64_t *node_count, const int32_t *entries, int64_t m,
                     const int32_t *perms, int32_t k, int32_t *order, int32_t *signature) {
  const int64_t INF = INT64_MAX;
  if (N < 1 || B < 1 || k < 1 || m < 0) return -1;
  /* each sample's node set, as a sorted array for membership tests */
  int32_t **set = (int32_t **)malloc((size_t)B * sizeof(int32_t *));
  for (int32_t i = 0; i < B; ++i) {
    set[i] = (int32_t *)malloc((size_t)(node_count[i] + 1) * sizeof(int32_t));
    memcpy(set[i], nodes + (int64_t)i * node_stride, (size_t)node_count[i] * sizeof(int32_t));
    qsort(set[i], (size_t)node_count[i], sizeof(int32_t), cmp_i32);
  }
  or_sig *sig = (or_sig *)malloc((size_t)(m + 1) * sizeof(or_sig));
  int rc = 0;
  for (int64_t e = 0; e < m && rc == 0; ++e) {
    int32_t v = entries[e];
    if (v < 0 || v >= N) { rc = -1; break; }
    int64_t s = INF;
    for (int32_t i = 0; i < B; ++i) {
      if (find_i32(set[i], node_count[i], v) < 0) continue; /* sample i does not require v */
      for (int32_t j = 0; j < k; ++j) {
        int64_t h = perms[(int64_t)j * B + i];
        if (h < s) s = h;
      }
    }
    sig[e].s = s;
    sig[e].pos = e;
  }
  if (rc == 0) {
    for (int64_t e = 0; e < m; ++e) signature[e] = sig[e].s == INF ? -1 : (int32_t)sig[e].s;
    qsort(sig, (size_t)m, sizeof(or_sig), cmp_sig);
    for (int64_t r = 0; r < m; ++r) order[r] = entries[sig[r].pos];
  }
  for (int32_t i = 0; i < B; ++i) free(set[i]);
  free(set);
  free(sig);
  return rc;
}
