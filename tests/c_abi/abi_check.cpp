// The C ABI used from C++ alone, with plain device pointers from hipMalloc and
// a HIP stream: no Python, no torch.  One group is sampled and packed by
// dg_sample_pack_group (the size query first, with no packed capacity), then
// assembled by dg_assemble_batches, and everything is copied back and checked
// on the host against what the header's contract fixes for any input:
//  - each batch's list starts with its seeds; each hop's segment is the set of
//    that hop's sampled neighbours not listed before, ascending;
//  - every edge runs from a node of the previous segment to one of its CSR
//    neighbours; each frontier node has min(degree, fan-out) edges, to distinct
//    neighbours in ascending CSR order, and a node of degree <= fan-out has all
//    of them;
//  - P_b = the non-cached nodes of batch b, ascending; each packed row holds
//    the feature row of its node; the address tables point at the right cache
//    or packed row; each assembled row equals the feature row of its node;
//  - the membership words are left all-zero, and a null argument is rejected
//    with DG_EINVAL and a message;
//  - dg_sample_group followed by dg_pack_group (the two calls the one call
//    stands for) gives the same outputs on new buffers.
// Exit status 0 when every check holds.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <set>
#include <vector>

#include "dg.h"

#define HIP_OK(x)                                                            \
  do {                                                                       \
    hipError_t e_ = (x);                                                     \
    if (e_ != hipSuccess) {                                                  \
      std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), \
                   __LINE__);                                                \
      return 2;                                                              \
    }                                                                        \
  } while (0)

static int failures = 0;
#define CHECK(cond, ...)                     \
  do {                                       \
    if (!(cond)) {                           \
      if (failures < 20) {                   \
        std::fprintf(stderr, "FAIL: ");      \
        std::fprintf(stderr, __VA_ARGS__);   \
        std::fprintf(stderr, "\n");          \
      }                                      \
      ++failures;                            \
    }                                        \
  } while (0)

template <typename T>
static T *dev_alloc(size_t n) {
  void *p = nullptr;
  if (hipMalloc(&p, n * sizeof(T) > 0 ? n * sizeof(T) : 1) != hipSuccess) return nullptr;
  return static_cast<T *>(p);
}

int main() {
  // A graph of N nodes: node v has a degree of 0..23 and distinct sorted
  // neighbours other than itself, from a fixed integer recurrence.
  const int64_t N = 20000;
  std::vector<int64_t> off(N + 1, 0);
  std::vector<int32_t> idx;
  for (int64_t v = 0; v < N; ++v) {
    const int d = (int)(((uint64_t)v * 2654435761ull >> 7) % 24);
    std::set<int32_t> row;
    uint64_t x = (uint64_t)v * 6364136223846793005ull + 1442695040888963407ull;
    while ((int)row.size() < d) {
      x = x * 6364136223846793005ull + 1442695040888963407ull;
      const int32_t u = (int32_t)((x >> 33) % (uint64_t)N);
      if (u != v) row.insert(u);
    }
    idx.insert(idx.end(), row.begin(), row.end());
    off[v + 1] = (int64_t)idx.size();
  }
  const int64_t E = (int64_t)idx.size();
  const int32_t B = 8, S = 32, K = 3;
  const int32_t fan[K] = {6, 4, 3};
  std::vector<int32_t> seeds((size_t)B * S);
  for (int b = 0; b < B; ++b)
    for (int s = 0; s < S; ++s) seeds[(size_t)b * S + s] = (int32_t)((b * 977 + s * 131) % N);
  // features: 64-byte rows; every 7th node cached, cache row v/7 = X[v]
  const int64_t R = 64;
  std::vector<uint8_t> X((size_t)N * R);
  for (int64_t v = 0; v < N; ++v)
    for (int64_t i = 0; i < R; ++i) X[(size_t)(v * R + i)] = (uint8_t)((v * 131 + i * 7) & 0xff);
  std::vector<int32_t> slot(N, -1);
  const int64_t C = (N + 6) / 7;
  std::vector<uint8_t> cache((size_t)C * R);
  for (int64_t v = 0; v < N; v += 7) {
    slot[v] = (int32_t)(v / 7);
    std::memcpy(&cache[(size_t)(v / 7) * R], &X[(size_t)v * R], R);
  }

  std::printf("%s; N=%lld E=%lld B=%d S=%d fan-outs %d,%d,%d\n", dg_version(), (long long)N,
              (long long)E, B, S, fan[0], fan[1], fan[2]);
  int64_t node_cap = 0, edge_cap = 0;
  if (dg_sample_bounds(N, E, S, fan, K, DG_SAMPLE_DIRECT, &node_cap, &edge_cap) != DG_OK) {
    std::fprintf(stderr, "dg_sample_bounds: %s\n", dg_last_error());
    return 1;
  }
  const size_t ws_bytes = dg_sample_workspace_bytes(N, B, node_cap, edge_cap, DG_SAMPLE_DIRECT);
  const size_t pws_bytes = dg_sample_pack_workspace_bytes(N, B, node_cap);
  if (ws_bytes == 0 || pws_bytes == 0) {
    std::fprintf(stderr, "workspace queries returned 0\n");
    return 1;
  }

  hipStream_t st;
  HIP_OK(hipStreamCreate(&st));
  int64_t *d_off = dev_alloc<int64_t>(N + 1);
  int32_t *d_idx = dev_alloc<int32_t>(E), *d_seeds = dev_alloc<int32_t>(seeds.size());
  int32_t *d_slot = dev_alloc<int32_t>(N);
  uint8_t *d_X = dev_alloc<uint8_t>(X.size()), *d_cache = dev_alloc<uint8_t>(cache.size());
  int32_t *d_nodes = dev_alloc<int32_t>((size_t)B * node_cap);
  int32_t *d_esrc = dev_alloc<int32_t>((size_t)B * edge_cap);
  int32_t *d_edst = dev_alloc<int32_t>((size_t)B * edge_cap);
  int32_t *d_loc = dev_alloc<int32_t>((size_t)B * node_cap);
  int64_t *d_pptr = dev_alloc<int64_t>(B + 1);
  uint64_t *d_mem = dev_alloc<uint64_t>(N);
  void *d_ws = dev_alloc<uint8_t>(ws_bytes), *d_pws = dev_alloc<uint8_t>(pws_bytes);
  if (!d_off || !d_idx || !d_seeds || !d_slot || !d_X || !d_cache || !d_nodes || !d_esrc ||
      !d_edst || !d_loc || !d_pptr || !d_mem || !d_ws || !d_pws) {
    std::fprintf(stderr, "hipMalloc failed\n");
    return 2;
  }
  HIP_OK(hipMemcpy(d_off, off.data(), off.size() * 8, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_idx, idx.data(), idx.size() * 4, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_seeds, seeds.data(), seeds.size() * 4, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_slot, slot.data(), slot.size() * 4, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_X, X.data(), X.size(), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_cache, cache.data(), cache.size(), hipMemcpyHostToDevice));
  HIP_OK(hipMemset(d_mem, 0xff, (size_t)N * 8));  // garbage: the call is told nothing

  const dg_csr g{N, E, d_off, d_idx};
  std::vector<int64_t> hop_ptr((size_t)B * (K + 2)), edge_ptr((size_t)B * (K + 1));
  std::vector<int64_t> pptr_host(B + 1);
  dg_sizes sz;
  // size query: no packed capacity
  int rc = dg_sample_pack_group(&g, d_seeds, B, S, 0, fan, K, 7, DG_SAMPLE_DIRECT, node_cap,
                                d_nodes, hop_ptr.data(), edge_cap, d_esrc, d_edst,
                                edge_ptr.data(), d_mem, d_slot, d_loc, d_X, R, 0, nullptr,
                                nullptr, d_pptr, pptr_host.data(), nullptr, 0, 0, d_ws,
                                ws_bytes, d_pws, pws_bytes, st, nullptr, &sz, nullptr);
  if (rc != DG_ECAPACITY && rc != DG_OK) {
    std::fprintf(stderr, "size query: status %d: %s\n", rc, dg_last_error());
    return 1;
  }
  const int64_t rows = sz.packed_rows, nu = sz.unique_nodes;
  std::printf("pairs %lld, edges %lld, packed rows %lld, |U| %lld\n", (long long)sz.total_nodes,
              (long long)sz.total_edges, (long long)rows, (long long)nu);
  uint8_t *d_packed = dev_alloc<uint8_t>((size_t)rows * R);
  int32_t *d_pids = dev_alloc<int32_t>(rows), *d_uniq = dev_alloc<int32_t>(nu);
  if (!d_packed || !d_pids || !d_uniq) return 2;
  rc = dg_sample_pack_group(&g, d_seeds, B, S, 0, fan, K, 7, DG_SAMPLE_DIRECT, node_cap, d_nodes,
                            hop_ptr.data(), edge_cap, d_esrc, d_edst, edge_ptr.data(), d_mem,
                            d_slot, d_loc, d_X, R, rows, d_packed, d_pids, d_pptr,
                            pptr_host.data(), d_uniq, nu, 0, d_ws, ws_bytes, d_pws, pws_bytes, st,
                            nullptr, &sz, nullptr);
  if (rc != DG_OK) {
    std::fprintf(stderr, "dg_sample_pack_group: status %d: %s\n", rc, dg_last_error());
    return 1;
  }
  // assembly of every batch into buffers of its own
  std::vector<int64_t> counts(B);
  int64_t nmax = 0;
  for (int b = 0; b < B; ++b) {
    counts[b] = hop_ptr[(size_t)b * (K + 2) + K + 1];
    nmax = std::max(nmax, counts[b]);
  }
  std::vector<void *> outs(B);
  for (int b = 0; b < B; ++b)
    if (!(outs[b] = dev_alloc<uint8_t>((size_t)nmax * R))) return 2;
  int32_t *d_status = dev_alloc<int32_t>(1);
  if (!d_status) return 2;
  HIP_OK(hipMemset(d_status, 0, 4));
  rc = dg_assemble_batches(d_cache, C, d_packed, pptr_host.data(), d_loc, node_cap, counts.data(),
                           B, R, outs.data(), B, d_status, st);
  if (rc != DG_OK) {
    std::fprintf(stderr, "dg_assemble_batches: status %d: %s\n", rc, dg_last_error());
    return 1;
  }
  HIP_OK(hipStreamSynchronize(st));

  // copy back
  std::vector<int32_t> nodes((size_t)B * node_cap), esrc((size_t)B * edge_cap),
      edst((size_t)B * edge_cap), loc((size_t)B * node_cap), pids(rows), uniq(nu);
  std::vector<uint8_t> packed((size_t)rows * R);
  std::vector<uint64_t> mem(N);
  std::vector<int64_t> pptr_dev(B + 1);
  int32_t status = -1;
  HIP_OK(hipMemcpy(nodes.data(), d_nodes, nodes.size() * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(esrc.data(), d_esrc, esrc.size() * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(edst.data(), d_edst, edst.size() * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(loc.data(), d_loc, loc.size() * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(pids.data(), d_pids, pids.size() * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(uniq.data(), d_uniq, uniq.size() * 4, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(packed.data(), d_packed, packed.size(), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(mem.data(), d_mem, mem.size() * 8, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(pptr_dev.data(), d_pptr, pptr_dev.size() * 8, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(&status, d_status, 4, hipMemcpyDeviceToHost));

  CHECK(status == 0, "assembly status %d", status);
  CHECK(pptr_dev == pptr_host, "packed_ptr on the device and the host differ");
  CHECK(std::all_of(mem.begin(), mem.end(), [](uint64_t w) { return w == 0; }),
        "membership words not left all-zero");
  std::set<int32_t> U, U_nc;
  int64_t pairs = 0, edges = 0;
  for (int b = 0; b < B; ++b) {
    const int32_t *nb = &nodes[(size_t)b * node_cap];
    const int64_t *hp = &hop_ptr[(size_t)b * (K + 2)];
    const int64_t *ep = &edge_ptr[(size_t)b * (K + 1)];
    const int64_t n = hp[K + 1];
    pairs += n;
    edges += ep[K];
    CHECK(hp[0] == 0 && hp[1] == S, "batch %d: seed segment [%lld, %lld)", b, (long long)hp[0],
          (long long)hp[1]);
    for (int s = 0; s < S; ++s) CHECK(nb[s] == seeds[(size_t)b * S + s], "batch %d seed %d", b, s);
    std::set<int32_t> listed(nb, nb + S);
    for (int k = 1; k <= K; ++k) {
      // hop k: edges from segment k-1 to neighbours; the new ones form segment k
      std::set<int32_t> reached;
      int64_t prev_src = -1, prev_pos = -1;
      std::vector<int> per_src(n, 0);
      for (int64_t e = ep[k - 1]; e < ep[k]; ++e) {
        const int32_t s = esrc[(size_t)b * edge_cap + e], d = edst[(size_t)b * edge_cap + e];
        CHECK(s >= hp[k - 1] && s < hp[k], "batch %d hop %d: edge source %d outside the frontier",
              b, k, s);
        CHECK(d >= 0 && d < n, "batch %d hop %d: edge target %d outside the list", b, k, d);
        if (!(s >= 0 && s < n && d >= 0 && d < n)) continue;
        const int32_t v = nb[s], u = nb[d];
        const int32_t *r0 = &idx[(size_t)off[v]], *r1 = &idx[(size_t)off[v + 1]];
        const int32_t *at = std::lower_bound(r0, r1, u);
        CHECK(at != r1 && *at == u, "batch %d hop %d: %d -> %d is not a graph edge", b, k, v, u);
        const int64_t pos = at - r0;
        if (s == prev_src) CHECK(pos > prev_pos, "batch %d hop %d: node %d's draws not ascending", b, k, v);
        CHECK(s >= prev_src, "batch %d hop %d: edges not in frontier order", b, k);
        prev_src = s;
        prev_pos = pos;
        ++per_src[s];
        if (!listed.count(u)) reached.insert(u);
      }
      for (int64_t s = hp[k - 1]; s < hp[k]; ++s) {
        const int64_t deg = off[nb[s] + 1] - off[nb[s]];
        CHECK(per_src[s] == std::min<int64_t>(deg, fan[k - 1]),
              "batch %d hop %d: node %d has %d edges, degree %lld", b, k, nb[s], per_src[s],
              (long long)deg);
      }
      const std::vector<int32_t> seg(nb + hp[k], nb + hp[k + 1]);
      const std::vector<int32_t> want(reached.begin(), reached.end());
      CHECK(seg == want, "batch %d hop %d: segment of %zu nodes, %zu new neighbours", b, k,
            seg.size(), want.size());
      listed.insert(seg.begin(), seg.end());
    }
    CHECK((int64_t)listed.size() == n, "batch %d: a node listed twice", b);
    // packing: P_b, packed rows, address tables
    std::vector<int32_t> Pb;
    for (int64_t j = 0; j < n; ++j) {
      U.insert(nb[j]);
      if (slot[nb[j]] < 0) Pb.push_back(nb[j]);
    }
    std::sort(Pb.begin(), Pb.end());
    for (int32_t u : Pb) U_nc.insert(u);
    const int64_t p0 = pptr_host[b], p1 = pptr_host[b + 1];
    CHECK(p1 - p0 == (int64_t)Pb.size(), "batch %d: %lld packed rows, %zu non-cached nodes", b,
          (long long)(p1 - p0), Pb.size());
    if (p1 - p0 == (int64_t)Pb.size())
      for (int64_t r = 0; r < p1 - p0; ++r) {
        CHECK(pids[p0 + r] == Pb[r], "batch %d packed row %lld holds node %d, want %d", b,
              (long long)r, pids[p0 + r], Pb[r]);
        CHECK(std::memcmp(&packed[(size_t)(p0 + r) * R], &X[(size_t)Pb[r] * R], R) == 0,
              "batch %d packed row %lld: wrong bytes", b, (long long)r);
      }
    std::vector<uint8_t> y((size_t)n * R);
    HIP_OK(hipMemcpy(y.data(), outs[b], y.size(), hipMemcpyDeviceToHost));
    for (int64_t j = 0; j < n; ++j) {
      const int32_t u = nb[j], l = loc[(size_t)b * node_cap + j];
      if (slot[u] >= 0) {
        CHECK(l == -(slot[u] + 1), "batch %d entry %lld: loc %d for cached node %d", b,
              (long long)j, l, u);
      } else {
        CHECK(l >= 0 && l < p1 - p0 && pids[p0 + l] == u, "batch %d entry %lld: loc %d", b,
              (long long)j, l);
      }
      CHECK(std::memcmp(&y[(size_t)j * R], &X[(size_t)u * R], R) == 0,
            "batch %d assembled row %lld: wrong bytes", b, (long long)j);
    }
  }
  CHECK(sz.total_nodes == pairs && sz.total_edges == edges, "sizes disagree with the lists");
  CHECK(sz.unique_nodes == (int64_t)U.size() && sz.unique_packed == (int64_t)U_nc.size(),
        "|U| %lld / %zu, |U_nc| %lld / %zu", (long long)sz.unique_nodes, U.size(),
        (long long)sz.unique_packed, U_nc.size());
  CHECK(std::vector<int32_t>(U.begin(), U.end()) == uniq, "group_unique is not U, ascending");

  // The same group by the two calls the one call stands for: dg_sample_group
  // (membership words and the cached nodes' address-table entries) followed by
  // dg_pack_group (clearing the words, completing the pending entries), on new
  // buffers; every output must equal the one call's.
  {
    const size_t ws2_bytes = dg_sample_workspace_bytes(N, B, node_cap, edge_cap, DG_SAMPLE_DIRECT);
    const size_t pws2_bytes = dg_pack_workspace_bytes(N, B, pairs);
    int32_t *n2 = dev_alloc<int32_t>((size_t)B * node_cap);
    int32_t *es2 = dev_alloc<int32_t>((size_t)B * edge_cap), *ed2 = dev_alloc<int32_t>((size_t)B * edge_cap);
    int32_t *loc2 = dev_alloc<int32_t>((size_t)B * node_cap);
    uint8_t *pk2 = dev_alloc<uint8_t>((size_t)rows * R);
    int32_t *pid2 = dev_alloc<int32_t>(rows), *uq2 = dev_alloc<int32_t>(nu);
    int64_t *pp2 = dev_alloc<int64_t>(B + 1);
    void *ws2 = dev_alloc<uint8_t>(ws2_bytes), *pws2 = dev_alloc<uint8_t>(pws2_bytes);
    if (!n2 || !es2 || !ed2 || !loc2 || !pk2 || !pid2 || !uq2 || !pp2 || !ws2 || !pws2 ||
        ws2_bytes == 0 || pws2_bytes == 0) {
      std::fprintf(stderr, "two-call buffers: allocation or query failed\n");
      return 2;
    }
    std::vector<int64_t> hp2((size_t)B * (K + 2)), ep2((size_t)B * (K + 1)), pph2(B + 1);
    dg_sizes s2, p2;
    rc = dg_sample_group(&g, d_seeds, B, S, 0, fan, K, 7, DG_SAMPLE_DIRECT, node_cap, n2,
                         hp2.data(), edge_cap, es2, ed2, ep2.data(), d_mem, nullptr, d_slot, loc2,
                         ws2, ws2_bytes, st, &s2, nullptr);
    CHECK(rc == DG_OK, "dg_sample_group: status %d: %s", rc, dg_last_error());
    rc = dg_pack_group(d_X, N, R, d_slot, B, n2, node_cap, counts.data(), rows, pk2, pid2, pp2,
                       pph2.data(), loc2, uq2, nu, d_mem, nullptr, nullptr, 0, nullptr,
                       DG_PACK_CLEAR_MEMBERSHIP | DG_PACK_LOC_PENDING, pws2, pws2_bytes, st,
                       nullptr, &p2, nullptr);
    CHECK(rc == DG_OK, "dg_pack_group: status %d: %s", rc, dg_last_error());
    HIP_OK(hipStreamSynchronize(st));
    CHECK(hp2 == hop_ptr && ep2 == edge_ptr && pph2 == pptr_host, "two calls: bounds differ");
    CHECK(p2.packed_rows == rows && p2.unique_nodes == nu && p2.unique_packed == sz.unique_packed,
          "two calls: packing sizes differ");
    auto same = [&](const void *d, const void *h, size_t bytes) {
      std::vector<uint8_t> t(bytes);
      if (hipMemcpy(t.data(), d, bytes, hipMemcpyDeviceToHost) != hipSuccess) return false;
      return bytes == 0 || std::memcmp(t.data(), h, bytes) == 0;
    };
    for (int b = 0; b < B; ++b) {
      const int64_t n = counts[b], e = edge_ptr[(size_t)b * (K + 1) + K];
      const size_t o = (size_t)b * node_cap, oe = (size_t)b * edge_cap;
      CHECK(same(n2 + o, &nodes[o], (size_t)n * 4), "two calls: batch %d nodes differ", b);
      CHECK(same(loc2 + o, &loc[o], (size_t)n * 4), "two calls: batch %d loc differs", b);
      CHECK(same(es2 + oe, &esrc[oe], (size_t)e * 4) && same(ed2 + oe, &edst[oe], (size_t)e * 4),
            "two calls: batch %d edges differ", b);
    }
    CHECK(same(pid2, pids.data(), (size_t)rows * 4) && same(uq2, uniq.data(), (size_t)nu * 4),
          "two calls: packed_ids or U differ");
    CHECK(same(pk2, packed.data(), (size_t)rows * R), "two calls: packed rows differ");
    std::vector<uint64_t> m2(N);
    HIP_OK(hipMemcpy(m2.data(), d_mem, (size_t)N * 8, hipMemcpyDeviceToHost));
    CHECK(std::all_of(m2.begin(), m2.end(), [](uint64_t w) { return w == 0; }),
          "two calls: membership words not left all-zero");
  }

  // a null argument is rejected before any work, with a message
  rc = dg_sample_pack_group(&g, nullptr, B, S, 0, fan, K, 7, DG_SAMPLE_DIRECT, node_cap, d_nodes,
                            hop_ptr.data(), edge_cap, d_esrc, d_edst, edge_ptr.data(), d_mem,
                            d_slot, d_loc, d_X, R, rows, d_packed, d_pids, d_pptr,
                            pptr_host.data(), d_uniq, nu, 0, d_ws, ws_bytes, d_pws, pws_bytes, st,
                            nullptr, &sz, nullptr);
  CHECK(rc == DG_EINVAL && std::strlen(dg_last_error()) > 0, "null seeds: status %d", rc);

  HIP_OK(hipDeviceSynchronize());
  if (failures) {
    std::fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  std::printf("C ABI check ok: %lld pairs, %lld edges, %lld packed rows\n", (long long)pairs,
              (long long)edges, (long long)rows);
  return 0;
}
