"""Pins for the CPU oracle: each test ties it to something other than itself —
the paper's worked examples, published generator outputs, closed forms,
brute-force set computations on tiny inputs, the breadth-first-search special
case and chi-square uniformity.  CPU only."""
import itertools
import json
import os
import random
from collections import deque

import numpy as np
import pytest

from conftest import GOLDEN

M64 = 2**64 - 1


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def csr_from_rows(n, rows):
    off = np.zeros(n + 1, dtype=np.int64)
    idx = []
    for v in range(n):
        r = rows.get(str(v), rows.get(v, []))
        idx.extend(r)
        off[v + 1] = off[v] + len(r)
    return off, np.array(idx, dtype=np.int32)


# ------------------------------------------------------------------ RNG pins
def test_splitmix64_published_outputs(orc):
    """The mixer is SplitMix64's output function: reproduce the published
    next() sequence (state += gamma, output mix(state))."""
    fx = load("splitmix64.json")
    for seq in fx["sequences"]:
        for i, want in enumerate(seq["outputs"]):
            assert orc.splitmix_nth(seq["seed"], i) == int(want, 0)


def test_below_closed_forms(orc):
    for m in (1, 2, 3, 7, 10, 1000, 2**31 - 1, 2**40 + 3):
        assert orc.below(0, m) == 0
        assert orc.below(M64, m) == m - 1
    for k in (1, 5, 1 << 20):
        assert orc.below(1 << 63, 2 * k) == k          # half-way point
    for h in (0, 12345, 1 << 63, M64):
        assert orc.below(h, 1) == 0
        assert orc.below(h, 1 << 32) == h >> 32        # power of two: top bits
    hs = sorted(random.Random(1).getrandbits(64) for _ in range(200))
    vals = [orc.below(h, 97) for h in hs]
    assert vals == sorted(vals)                        # monotone in h


# ------------------------------------------------------------------ Floyd pins
def test_floyd_basic_properties(orc):
    rnd = random.Random(7)
    for _ in range(300):
        d = rnd.randint(0, 60)
        f = rnd.randint(0, d)
        got = orc.floyd(d, f, rnd.getrandbits(64))
        assert len(got) == f
        assert got == sorted(set(got))
        assert all(0 <= x < d for x in got)
    assert orc.floyd(9, 9, 123) == list(range(9))
    assert orc.floyd(9, 0, 123) == []


def _chi2_ok(counts, expected, dof):
    # chi-square statistic against a generous bound (mean dof, sd sqrt(2 dof))
    stat = sum((c - expected) ** 2 / expected for c in counts)
    return stat < dof + 6 * (2 * dof) ** 0.5, stat


def test_floyd_subsets_uniform(orc):
    """All C(5,2) = 10 subsets equally likely over many keys."""
    n = 60000
    counts = {s: 0 for s in itertools.combinations(range(5), 2)}
    for g in range(n):
        key = orc.draw_key(99, g, 1, 4)
        counts[tuple(orc.floyd(5, 2, key))] += 1
    ok, stat = _chi2_ok(list(counts.values()), n / 10, 9)
    assert ok, stat


def test_floyd_inclusion_probability(orc):
    """Each position is included with probability f/d."""
    d, f, n = 40, 7, 20000
    hits = np.zeros(d)
    for g in range(n):
        hits[orc.floyd(d, f, orc.draw_key(5, g, 2, 11))] += 1
    ok, stat = _chi2_ok(hits.tolist(), n * f / d, d - 1)
    assert ok, stat


def test_draw_key_separates_batch_hop_node(orc):
    """Changing the batch, the hop or the node gives an independent subset:
    two draws agree on a 2-of-5 subset about 1/10 of the time, not always."""
    n = 20000
    for vary in ("g", "k", "v"):
        same = 0
        for t in range(n):
            a = orc.draw_key(3, t, 1, 77)
            b = orc.draw_key(3, t + 1 if vary == "g" else t, 2 if vary == "k" else 1,
                             78 if vary == "v" else 77)
            same += orc.floyd(5, 2, a) == orc.floyd(5, 2, b)
        assert abs(same / n - 0.1) < 0.015, (vary, same / n)


# ------------------------------------------------------------------ paper examples
def test_fig1_worked_example(orc):
    fx = load("fig1_sampling.json")
    off, idx = csr_from_rows(fx["num_nodes"], fx["rows"])
    r = orc.sample_group(off, idx, np.array(fx["seeds"], dtype=np.int32), fx["fanouts"], 0)
    ex = fx["expect"]
    nodes = r["nodes"][0]
    assert nodes.tolist() == ex["nodes"]
    assert r["hop_ptr"][0].tolist() == ex["hop_ptr"]
    assert r["edge_ptr"][0].tolist() == ex["edge_ptr"]
    edges = [[int(nodes[s]), int(nodes[d])] for s, d in zip(r["edge_src"][0], r["edge_dst"][0])]
    assert edges == ex["edges_global"]


def test_fig1_worked_example_layered(orc):
    """Layer-wise variant: at step 2 the seed samples again (its two neighbours
    are already in the mini-batch), so hop 2 repeats (v0,v3),(v0,v5) and the
    node list is unchanged."""
    fx = load("fig1_sampling.json")
    off, idx = csr_from_rows(fx["num_nodes"], fx["rows"])
    r = orc.sample_group(off, idx, np.array(fx["seeds"], dtype=np.int32), fx["fanouts"], 0,
                         layered=True)
    nodes = r["nodes"][0]
    assert nodes.tolist() == fx["expect"]["nodes"]
    edges = [[int(nodes[s]), int(nodes[d])] for s, d in zip(r["edge_src"][0], r["edge_dst"][0])]
    assert edges == [[0, 3], [0, 5], [0, 3], [0, 5], [3, 2], [3, 7], [5, 9], [5, 11]]
    assert r["edge_ptr"][0].tolist() == [0, 2, 8]


def test_fig3_worked_example(orc):
    fx = load("fig3_assembling.json")
    n = fx["num_nodes"]
    X = (np.arange(n, dtype=np.int32)[:, None] * 10 + np.arange(4, dtype=np.int32)[None, :])
    slot = np.full(n, -1, dtype=np.int32)
    for v, s in fx["cache_slots"].items():
        slot[int(v)] = s
    cache_nodes = sorted(fx["cache_slots"], key=lambda v: fx["cache_slots"][v])
    cache = X[[int(v) for v in cache_nodes]]
    req = np.array(fx["required"], dtype=np.int32)
    p = orc.pack_group(X, slot, [req])
    ex = fx["expect"]
    assert p["packed_ids"].tolist() == ex["packed_ids"]
    assert p["loc"][0].tolist() == ex["loc"]
    y = orc.assemble_batch(cache, p["packed"], p["loc"][0], X.shape[1] * 4)
    assert np.array_equal(y.view(np.int32), X[ex["assembled_nodes"]])


def test_fig6_worked_example(orc):
    fx = load("fig6_packing.json")
    n = fx["num_nodes"]
    X = np.arange(n * 3, dtype=np.float32).reshape(n, 3) + 0.5
    slot = np.full(n, -1, dtype=np.int32)
    for case in fx["cases"]:
        p = orc.pack_group(X, slot, [np.array(b, dtype=np.int32) for b in case["batches"]])
        ex = case["expect"]
        assert p["packed_ids"].tolist() == ex["packed_ids"], case["name"]
        assert p["packed_ptr"].tolist() == ex["packed_ptr"]
        assert p["unique"].tolist() == ex["unique"]
        assert [x.tolist() for x in p["loc"]] == ex["loc"]
        assert p["unique_packed"] == ex["unique_packed"]
        assert np.array_equal(p["packed"].view(np.float32), X[ex["packed_ids"]])


# ------------------------------------------------------------------ brute force
def random_csr(rnd, n, maxdeg):
    rows = {}
    for v in range(n):
        d = rnd.randint(0, min(maxdeg, n - 1))
        rows[v] = sorted(rnd.sample([u for u in range(n) if u != v], d))
    return csr_from_rows(n, rows), rows


def check_sample_invariants(rows, seeds, fanouts, r, layered=False):
    """Independent brute-force check of a sampling result (every rule except the
    identity of the random subset).  layered: every node so far samples at
    each hop, instead of only the previous hop's new nodes."""
    K = len(fanouts)
    for b, sd in enumerate(seeds):
        nodes = [int(x) for x in r["nodes"][b]]
        hop = r["hop_ptr"][b].tolist()
        ep = r["edge_ptr"][b].tolist()
        src = r["edge_src"][b].tolist()
        dst = r["edge_dst"][b].tolist()
        assert len(set(nodes)) == len(nodes)                      # unique
        assert nodes[:len(sd)] == [int(x) for x in sd]            # seeds first, in order
        assert hop[0] == 0 and hop[1] == len(sd) and hop[K + 1] == len(nodes)
        seen = set(nodes[:len(sd)])
        for k in range(1, K + 1):
            f = fanouts[k - 1]
            frontier = list(range(0 if layered else hop[k - 1], hop[k]))
            es = list(range(ep[k - 1], ep[k]))
            # parents: frontier positions, non-decreasing, each drawing min(d, f)
            parents = [src[e] for e in es]
            assert parents == sorted(parents)
            for p in frontier:
                v = nodes[p]
                mine = [e for e in es if src[e] == p]
                d = len(rows[v])
                want = d if (f < 0 or d <= f) else f
                assert len(mine) == want
                nbrs = [nodes[dst[e]] for e in mine]
                assert all(u in rows[v] for u in nbrs)                # real edges
                pos = [rows[v].index(u) for u in nbrs]
                assert pos == sorted(set(pos))                      # ascending, distinct
                if want == d:
                    assert nbrs == rows[v]
            assert set(parents) <= set(frontier)
            # the hop-k segment = new sampled neighbours, ascending
            sampled = {nodes[dst[e]] for e in es}
            new = sorted(sampled - seen)
            assert nodes[hop[k]:hop[k + 1]] == new
            seen |= set(new)
        assert ep[K] == len(src) == len(dst)
        assert all(0 <= x < len(nodes) for x in src + dst)


@pytest.mark.parametrize("layered", [False, True])
@pytest.mark.parametrize("trial", range(40))
def test_sampling_bruteforce(orc, trial, layered):
    rnd = random.Random(1000 + trial)
    n = rnd.randint(2, 40)
    (off, idx), rows = random_csr(rnd, n, rnd.choice([2, 5, 9]))
    B = rnd.randint(1, 4)
    S = rnd.randint(1, min(5, n))
    seeds = [rnd.sample(range(n), S) for _ in range(B)]
    K = rnd.randint(0, 3)
    fan = [rnd.choice([-1, 0, 1, 2, 3, 5]) for _ in range(K)]
    r = orc.sample_group(off, idx, np.array(seeds, dtype=np.int32), fan, rnd.getrandbits(64),
                         batch_base=rnd.randint(0, 100), layered=layered)
    check_sample_invariants(rows, seeds, fan, r, layered)


def test_sampling_batches_independent(orc):
    """A group split into two calls (batch_base offsets) equals one call."""
    rnd = random.Random(3)
    (off, idx), rows = random_csr(rnd, 200, 12)
    seeds = np.array([rnd.sample(range(200), 6) for _ in range(5)], dtype=np.int32)
    whole = orc.sample_group(off, idx, seeds, [3, 2, 2], 42, batch_base=10)
    a = orc.sample_group(off, idx, seeds[:2], [3, 2, 2], 42, batch_base=10)
    b = orc.sample_group(off, idx, seeds[2:], [3, 2, 2], 42, batch_base=12)
    for key in ("nodes", "edge_src", "edge_dst", "hop_ptr", "edge_ptr"):
        for x, y in zip(whole[key], a[key] + b[key]):
            assert np.array_equal(x, y)


@pytest.mark.parametrize("layered", [False, True])
@pytest.mark.parametrize("trial", range(12))
def test_bfs_special_case(orc, trial, layered):
    """With f < 0 (or f >= max degree) sampling is deterministic and the node
    list is the seeds followed by the breadth-first layers, each ascending."""
    rnd = random.Random(50 + trial)
    n = rnd.randint(5, 60)
    (off, idx), rows = random_csr(rnd, n, 6)
    S = rnd.randint(1, 4)
    seeds = rnd.sample(range(n), S)
    K = rnd.randint(1, 4)
    fan = [rnd.choice([-1, 6, 100]) for _ in range(K)]
    r = orc.sample_group(off, idx, np.array([seeds], dtype=np.int32), fan, 1, layered=layered)
    dist = {s: 0 for s in seeds}
    q = deque(seeds)
    while q:
        v = q.popleft()
        for u in rows[v]:
            if u not in dist:
                dist[u] = dist[v] + 1
                q.append(u)
    want = list(seeds)
    for k in range(1, K + 1):
        want += sorted(u for u, d in dist.items() if d == k)
    assert r["nodes"][0].tolist() == want
    if layered:  # hop k: every node within distance k-1 samples all its neighbours
        frontier_edges = sum(len(rows[v]) * (K - d) for v, d in dist.items() if d < K)
    else:
        frontier_edges = sum(len(rows[v]) for v, d in dist.items() if d < K)
    assert r["edge_ptr"][0][K] == frontier_edges


# ------------------------------------------------------------------ packing / assembly
@pytest.mark.parametrize("trial", range(25))
def test_pack_assemble_bruteforce(orc, trial):
    rnd = random.Random(500 + trial)
    n = rnd.randint(1, 80)
    R = rnd.choice([1, 3, 4, 16, 24])
    X = np.frombuffer(rnd.randbytes(n * R), dtype=np.uint8).reshape(n, R).copy()
    ncache = rnd.randint(0, n)
    cache_nodes = rnd.sample(range(n), ncache)
    slot = np.full(n, -1, dtype=np.int32)
    for s, v in enumerate(cache_nodes):
        slot[v] = s
    cache = X[cache_nodes] if ncache else np.zeros((0, R), dtype=np.uint8)
    B = rnd.randint(1, 6)
    lists = [np.array(rnd.sample(range(n), rnd.randint(0, n)), dtype=np.int32) for _ in range(B)]
    p = orc.pack_group(X, slot, lists)
    U = sorted(set().union(*[set(x.tolist()) for x in lists]))
    assert p["unique"].tolist() == U
    assert p["unique_packed"] == sum(1 for u in U if slot[u] < 0)
    ptr = [0]
    for b, lst in enumerate(lists):
        Pb = sorted(u for u in lst.tolist() if slot[u] < 0)
        assert p["packed_ids"][ptr[-1]:ptr[-1] + len(Pb)].tolist() == Pb
        ptr.append(ptr[-1] + len(Pb))
        for j, u in enumerate(lst.tolist()):
            l = int(p["loc"][b][j])
            if slot[u] >= 0:
                assert l == -(int(slot[u]) + 1)
            else:
                assert Pb[l] == u
        chunk = p["packed"][ptr[b]:ptr[b + 1]]
        y = orc.assemble_batch(cache, chunk, p["loc"][b], R)
        assert np.array_equal(y, X[lst]) if len(lst) else y.shape[0] == 0
    assert p["packed_ptr"].tolist() == ptr
    assert np.array_equal(p["packed"], X[p["packed_ids"]])


def test_pack_rejects_bad_lists(orc):
    X = np.zeros((5, 4), dtype=np.uint8)
    slot = np.full(5, -1, dtype=np.int32)
    with pytest.raises(orc.OracleError):
        orc.pack_group(X, slot, [np.array([1, 1], dtype=np.int32)])
    with pytest.raises(orc.OracleError):
        orc.pack_group(X, slot, [np.array([5], dtype=np.int32)])


def test_sample_rejects_duplicate_seed(orc):
    off, idx = csr_from_rows(3, {0: [1], 1: [2], 2: [0]})
    with pytest.raises(orc.OracleError):
        orc.sample_group(off, idx, np.array([[1, 1]], dtype=np.int32), [1], 0)


# ------------------------------------------------------------------ access-frequency cache
def packed_volume(slot, lists):
    return sum(int((slot[np.asarray(l, dtype=np.int64)] < 0).sum()) for l in lists)


@pytest.mark.parametrize("trial", range(20))
def test_cache_by_frequency_bruteforce_and_optimal(orc, trial):
    """Counts = number of lists holding the node; ranking count-descending,
    ID-ascending; and (the placement claim of §3) no other cache of the same
    size leaves fewer rows to pack."""
    rnd = random.Random(700 + trial)
    n = rnd.randint(1, 60)
    B = rnd.randint(1, 6)
    lists = [np.array(rnd.sample(range(n), rnd.randint(0, n)), dtype=np.int32) for _ in range(B)]
    C = rnd.randint(0, n)
    slot, nodes, cached = orc.cache_by_frequency(n, lists, C)
    count = {u: sum(u in set(l.tolist()) for l in lists) for u in range(n)}
    want = sorted((u for u in range(n) if count[u] > 0), key=lambda u: (-count[u], u))[:C]
    assert nodes[:len(want)].tolist() == want and cached == len(want)
    assert all(x == -1 for x in nodes[len(want):].tolist())
    assert [int(slot[u]) for u in want] == list(range(len(want)))
    assert sum(int(s >= 0) for s in slot) == len(want)
    best = packed_volume(slot, lists)
    for _ in range(30):
        other = np.full(n, -1, dtype=np.int32)
        for s, u in enumerate(rnd.sample(range(n), min(C, n))):
            other[u] = s
        assert best <= packed_volume(other, lists)


def test_cache_by_frequency_small_example(orc):
    # node 2 in three lists, 0 and 5 in two, 7 in one
    lists = [np.array(x, dtype=np.int32) for x in ([2, 0, 7], [5, 2], [0, 2, 5])]
    slot, nodes, cached = orc.cache_by_frequency(8, lists, 3)
    assert nodes.tolist() == [2, 0, 5] and cached == 3
    slot, nodes, cached = orc.cache_by_frequency(8, lists, 6)
    assert nodes.tolist() == [2, 0, 5, 7, -1, -1] and cached == 4


# ------------------------------------------------------------------ MinHash reordering
@pytest.mark.parametrize("trial", range(20))
def test_minhash_order_matches_set_definition(orc, trial):
    """S(v) is the classic MinHash of v's sample set under each permutation
    (the minimum permuted sample ID), minimised over the k permutations;
    entries are stably sorted by it, samples-less entries last."""
    rnd = random.Random(900 + trial)
    n = rnd.randint(1, 50)
    B = rnd.randint(1, 8)
    lists = [np.array(rnd.sample(range(n), rnd.randint(0, n)), dtype=np.int32) for _ in range(B)]
    m = rnd.randint(0, n)
    entries = np.array(rnd.sample(range(n), m), dtype=np.int32)
    k = rnd.randint(1, 4)
    perms = np.array([rnd.sample(range(B), B) for _ in range(k)], dtype=np.int32)
    order, sig = orc.minhash_order(n, lists, entries, perms)
    samples = {v: {i for i in range(B) if v in set(lists[i].tolist())} for v in range(n)}
    want_sig = []
    for v in entries.tolist():
        per_perm = [min((int(p[i]) for i in samples[v]), default=None) for p in perms]
        want_sig.append(-1 if not samples[v] else min(per_perm))
    assert sig.tolist() == want_sig
    key = [(s if s >= 0 else 10**9, pos) for pos, s in enumerate(want_sig)]
    want_order = [int(entries[pos]) for _, pos in sorted(key)]
    assert order.tolist() == want_order


def test_minhash_order_groups_nodes_with_equal_sample_sets(orc):
    # nodes 1 and 6 are required by samples {0, 2}; 3 and 4 by {1}; 5 by none
    lists = [np.array(x, dtype=np.int32) for x in ([1, 6, 2], [3, 4, 2], [6, 1])]
    entries = np.array([1, 3, 5, 6, 4], dtype=np.int32)
    perms = np.array([[2, 0, 1], [1, 2, 0]], dtype=np.int32)
    order, sig = orc.minhash_order(8, lists, entries, perms)
    # samples {0,2}: min(2,1) under perm 0 -> 1, under perm 1 -> min(1,0) = 0  => S = 0
    # sample {1}:   perm 0 -> 0, perm 1 -> 2                                  => S = 0
    assert sig.tolist() == [0, 0, -1, 0, 0]
    assert order.tolist() == [1, 3, 6, 4, 5]
