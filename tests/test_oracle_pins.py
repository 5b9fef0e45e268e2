"""Pins for the CPU oracle (no GPU).

The paper prints no calling-context-tree values, so the oracle is pinned to what the
definition and mathematics fix: hand-worked trees (tests/golden), brute-force prefix
enumeration in two independent implementations (C++ std::set and pure Python tuple
sorting), closed forms for special shapes, algebraic laws, and an invariant checker
that is itself shown to catch planted mistakes.
"""
import math

import numpy as np
import pytest

import oracle
import tracegen
from conftest import load_golden

FIELDS = ("parent", "frame", "depth", "excl", "incl")


def assert_tree_equal(a, b, ctx=""):
    for k in FIELDS:
        x, y = np.asarray(a[k]), np.asarray(b[k])
        assert x.shape == y.shape, f"{ctx}: {k} shape {x.shape} vs {y.shape}"
        assert np.array_equal(x, y), f"{ctx}: {k} differs at {np.flatnonzero((x != y).ravel())[:5]}"


def py_brute(offsets, frames, metrics):
    """Independent pure-Python definition: nodes = distinct prefixes sorted as tuples
    (Python orders tuples lexicographically, a proper prefix first; ints compare as
    unsigned here because the frames are non-negative Python ints)."""
    n = len(offsets) - 1
    m = metrics.shape[1]
    paths = [tuple(int(x) for x in frames[offsets[i]:offsets[i + 1]]) for i in range(n)]
    nodes = sorted({p[:k] for p in paths for k in range(len(p) + 1)} | {()})
    idx = {p: i for i, p in enumerate(nodes)}
    mask = (1 << 64) - 1
    excl = [[0] * m for _ in nodes]
    incl = [[0] * m for _ in nodes]
    for i, p in enumerate(paths):
        for j in range(m):
            w = int(metrics[i, j])
            excl[idx[p]][j] = (excl[idx[p]][j] + w) & mask
            for k in range(len(p) + 1):
                incl[idx[p[:k]]][j] = (incl[idx[p[:k]]][j] + w) & mask
    return {
        "parent": np.array([0xFFFFFFFF if not p else idx[p[:-1]] for p in nodes], np.uint32),
        "frame": np.array([0 if not p else p[-1] for p in nodes], np.uint32),
        "depth": np.array([len(p) for p in nodes], np.uint32),
        "excl": np.array(excl, np.uint64).reshape(len(nodes), m),
        "incl": np.array(incl, np.uint64).reshape(len(nodes), m),
    }


@pytest.mark.parametrize("name", ["W1.txt", "W2.txt", "W3.txt", "W4.txt"])
def test_hand_worked(name):
    o, f, w, want = load_golden(name)
    got = oracle.build_tree(o, f, w)
    assert_tree_equal(got, want, name)
    assert_tree_equal(oracle.brute_tree(o, f, w), want, name + " brute")
    assert_tree_equal(py_brute(o, f, w), want, name + " py")
    assert oracle.check(got, oracle.total_metrics(w)) == (0, 0)


@pytest.mark.parametrize("seed", range(300))
def test_oracle_vs_brute_tiny_random(seed):
    # alphabet <= 4 and length <= 8 force shared prefixes, interior end nodes and
    # zero-length paths; metrics span the full uint64 range (wrap-around)
    n = 1 + seed % 60
    alphabet = 2 + seed % 3
    o, f, w = tracegen.random_small(n, alphabet, 8, 1 + seed % 3, seed)
    got = oracle.build_tree(o, f, w)
    assert_tree_equal(got, oracle.brute_tree(o, f, w), f"seed {seed}")
    assert oracle.check(got, oracle.total_metrics(w)) == (0, 0)


@pytest.mark.parametrize("seed", range(40))
def test_oracle_vs_python_definition(seed):
    o, f, w = tracegen.random_small(1 + seed % 30, 3 + seed % 6, 6, 2, 10_000 + seed)
    assert_tree_equal(oracle.build_tree(o, f, w), py_brute(o, f, w), f"seed {seed}")


def test_all_length_one_is_sort_unique_and_histogram():
    rng = np.random.default_rng(5)
    ids = np.array([0, 1, 0x7FFFFFFF, 0x80000000, 0xFFFFFFFF, 12345], np.uint32)
    f = ids[rng.integers(0, ids.size, 500)]
    o = np.arange(501, dtype=np.int64)
    w = rng.integers(0, 2**63, size=(500, 2), dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    t = oracle.build_tree(o, f, w)
    uniq = np.unique(f)  # numpy sorts uint32 as unsigned
    assert t.n_nodes == 1 + uniq.size
    assert np.array_equal(t["frame"][1:], uniq)
    assert np.all(t["parent"][1:] == 0) and np.all(t["depth"][1:] == 1)
    hist = np.zeros((uniq.size, 2), np.uint64)
    np.add.at(hist, np.searchsorted(uniq, f), w)  # uint64 adds wrap mod 2^64
    assert np.array_equal(t["excl"][1:], hist) and np.array_equal(t["incl"][1:], hist)
    assert np.array_equal(t["incl"][0], w.sum(axis=0, dtype=np.uint64))
    assert np.all(t["excl"][0] == 0)


@pytest.mark.parametrize("L", [1, 2, 7, 64, 512, 3000])
def test_single_path_is_a_chain(L):
    f = np.arange(L, dtype=np.uint32)[::-1].copy() * np.uint32(2654435761)
    o = np.array([0, L], np.int64)
    w = np.array([[123456789]], np.uint64)
    t = oracle.build_tree(o, f, w)
    assert t.n_nodes == L + 1
    assert np.array_equal(t["parent"][1:], np.arange(L, dtype=np.uint32))
    assert np.array_equal(t["frame"][1:], f)
    assert np.array_equal(t["depth"], np.arange(L + 1, dtype=np.uint32))
    assert np.all(t["incl"] == 123456789)
    assert np.all(t["excl"][:-1] == 0) and t["excl"][-1, 0] == 123456789


def test_all_events_identical():
    path = np.array([9, 3, 3, 9, 0xFFFFFFFF], np.uint32)
    n = 1000
    f = np.tile(path, n)
    o = np.arange(n + 1, dtype=np.int64) * path.size
    w = np.full((n, 1), 3, np.uint64)
    t = oracle.build_tree(o, f, w)
    assert t.n_nodes == path.size + 1
    assert np.all(t["incl"][:, 0] == 3 * n)
    assert t["excl"][-1, 0] == 3 * n and np.all(t["excl"][:-1] == 0)


def test_empty_input_is_root_only():
    t = oracle.build_tree(np.zeros(1, np.int64), np.zeros(0, np.uint32), np.zeros((0, 2), np.uint64))
    assert t.n_nodes == 1
    assert t["parent"][0] == 0xFFFFFFFF and np.all(t["excl"] == 0) and np.all(t["incl"] == 0)


def test_metrics_are_independent_columns():
    o, f, w = tracegen.random_paths(400, 20, 12, 4, seed=77)
    t = oracle.build_tree(o, f, w)
    for j in range(4):
        tj = oracle.build_tree(o, f, w[:, j:j + 1])
        for k in ("parent", "frame", "depth"):
            assert np.array_equal(t[k], tj[k])
        assert np.array_equal(t["excl"][:, j], tj["excl"][:, 0])
        assert np.array_equal(t["incl"][:, j], tj["incl"][:, 0])


def _subset(o, f, w, idx):
    lens = (o[1:] - o[:-1])[idx]
    oo = np.zeros(idx.size + 1, np.int64)
    oo[1:] = np.cumsum(lens)
    ff = np.concatenate([f[o[i]:o[i + 1]] for i in idx]) if idx.size else np.zeros(0, np.uint32)
    return oo, ff.astype(np.uint32), w[idx]


def test_permutation_invariance():
    o, f, w = tracegen.random_paths(500, 8, 10, 2, seed=3)
    perm = np.random.default_rng(0).permutation(500)
    assert_tree_equal(oracle.build_tree(o, f, w), oracle.build_tree(*_subset(o, f, w, perm)))


def test_incremental_ingest_equals_one_shot():
    o, f, w = tracegen.random_paths(900, 30, 16, 3, seed=11)
    one = oracle.build_tree(o, f, w)
    inc = oracle.Oracle(3)
    for a, b in [(0, 100), (100, 101), (101, 101), (101, 650), (650, 900)]:
        inc.ingest(*_subset(o, f, w, np.arange(a, b)))
    assert_tree_equal(one, inc.tree())


def test_exclusive_is_additive_over_a_split():
    o, f, w = tracegen.random_paths(600, 6, 8, 1, seed=21)
    idx = np.arange(600)
    a, b = idx[idx % 3 == 0], idx[idx % 3 != 0]
    t = oracle.build_tree(o, f, w)
    ta, tb = oracle.build_tree(*_subset(o, f, w, a)), oracle.build_tree(*_subset(o, f, w, b))

    def keyed(tr):
        # map root path -> excl via parent pointers
        paths = {0: ()}
        out = {}
        for v in range(1, tr.n_nodes):
            paths[v] = paths[int(tr["parent"][v])] + (int(tr["frame"][v]),)
        for v in range(tr.n_nodes):
            out[paths[v]] = int(tr["excl"][v, 0])
        return out
    ka, kb, kt = keyed(ta), keyed(tb), keyed(t)
    for p, e in kt.items():
        assert e == (ka.get(p, 0) + kb.get(p, 0)) % (1 << 64)


def test_point_query_matches_tree():
    o, f, w = tracegen.random_paths(300, 5, 7, 2, seed=8)
    t = oracle.build_tree(o, f, w)
    paths = {0: []}
    for v in range(1, t.n_nodes):
        paths[v] = paths[int(t["parent"][v])] + [int(t["frame"][v])]
    qs = list(range(t.n_nodes))
    qo = np.zeros(len(qs) + 1, np.int64)
    qo[1:] = np.cumsum([len(paths[v]) for v in qs])
    qf = np.array([x for v in qs for x in paths[v]], np.uint32)
    cnt, ex, inc = oracle.point_query(o, f, w, qo, qf, threads=2)
    assert np.all(cnt > 0)
    assert np.array_equal(ex, t["excl"]) and np.array_equal(inc, t["incl"])
    # a path that is not in the tree
    cnt, ex, inc = oracle.point_query(o, f, w, np.array([0, 2]), np.array([123456, 7], np.uint32))
    assert cnt[0] == 0 and np.all(inc == 0)


def test_malformed_offsets_rejected():
    with pytest.raises(ValueError):
        oracle.build_tree(np.array([1, 2]), np.zeros(2, np.uint32), np.zeros((1, 1), np.uint64))
    with pytest.raises(ValueError):
        oracle.build_tree(np.array([0, 3, 2]), np.zeros(3, np.uint32), np.zeros((2, 1), np.uint64))


# ---- the invariant checker catches planted mistakes (planted on the CPU, in oracle output)
def _good_tree():
    o, f, w = tracegen.random_paths(300, 6, 9, 2, seed=99)
    return oracle.build_tree(o, f, w), oracle.total_metrics(w)


def _plant(kind):
    t, tot = _good_tree()
    t = {k: v.copy() for k, v in t.items()}
    U = t["parent"].size
    if kind == "root":
        t["parent"][0] = 0
    elif kind == "parent_forward":
        t["parent"][5] = 7
    elif kind == "depth":
        t["depth"][9] += 1
    elif kind == "sibling_order":
        kids = np.flatnonzero(t["parent"] == 0)
        a, b = kids[0], kids[1]
        t["frame"][a], t["frame"][b] = t["frame"][b], t["frame"][a]
    elif kind == "not_preorder":
        # re-parent a node onto a finished subtree
        # W1's node [4] (id 5) re-parented under [1,2] (id 2, whose subtree ended at
        # id 3): depth and sibling order stay valid, only the preorder breaks
        o, f, w, _ = load_golden("W1.txt")
        t = {k: v.copy() for k, v in oracle.build_tree(o, f, w).items()}
        tot = oracle.total_metrics(w)
        t["parent"][5], t["depth"][5] = 2, 3
    elif kind == "dropped_child_term":
        v = int(np.flatnonzero(t["depth"] == 2)[0])
        t["incl"][v, 0] -= np.uint64(1)
    elif kind == "total":
        t["incl"][0, 1] += np.uint64(1)
        t["excl"][0, 1] += np.uint64(1)
    return t, tot


@pytest.mark.parametrize("kind,code", [("root", 1), ("parent_forward", 2), ("depth", 3),
                                       ("sibling_order", 4), ("not_preorder", 5),
                                       ("dropped_child_term", 6), ("total", 7)])
def test_checker_catches_planted_mistakes(kind, code):
    t, tot = _plant(kind)
    got, _ = oracle.check(t, tot)
    assert got == code, f"{kind}: expected code {code}, got {got}"


def test_checker_passes_workload_trees():
    for name in ("tiny", "layered_1m"):
        n = None if name == "tiny" else 100_000
        o, f, w = tracegen.generate(name, n_events=n)
        t = oracle.build_tree(o, f, w)
        assert oracle.check(t, oracle.total_metrics(w)) == (0, 0)


# ---- correlation-ID join (the flush step) -------------------------------------------
# Registry: ID 100 -> [5, 7], ID 7 -> [5, 9, 2], ID 3 -> [] (the empty path).
# Records (ID, metric): (7, 10), (999, 1), (100, 4), (7, 6), (3, 2).  By hand: record 1
# names no registered path; the others become, in record order, the events
# [5, 9, 2]:10, [5, 7]:4, [5, 9, 2]:6, []:2.  Their tree, by hand (ids = preorder of the
# prefixes (), (5), (5,7), (5,9), (5,9,2)): exclusive 2 / 0 / 4 / 0 / 16 and inclusive
# 22 / 20 / 4 / 16 / 16.
def test_join_hand_worked():
    o, f, w, unmatched = oracle.join_activity([0, 2, 5, 5], [5, 7, 5, 9, 2], [100, 7, 3], [7, 999, 100, 7, 3],
                                              [[10], [1], [4], [6], [2]])
    assert unmatched == 1
    assert o.tolist() == [0, 3, 5, 8, 8]
    assert f.tolist() == [5, 9, 2, 5, 7, 5, 9, 2]
    assert w.ravel().tolist() == [10, 4, 6, 2]
    t = oracle.build_tree(o, f, w)
    assert t["parent"].tolist() == [oracle.NO_PARENT, 0, 1, 1, 3]
    assert t["frame"].tolist() == [0, 5, 7, 9, 2]
    assert t["excl"].ravel().tolist() == [2, 0, 4, 0, 16]
    assert t["incl"].ravel().tolist() == [22, 20, 4, 16, 16]


def test_join_rejects_a_repeated_id():
    with pytest.raises(ValueError):
        oracle.join_activity([0, 1, 2], [1, 2], [5, 5], [5], [[1]])


def test_join_of_self_registered_events_is_the_trace():
    # every event registered under its own ID and flushed once, records shuffled: the
    # joined batch holds the trace's events (in another order), so the tree is the
    # trace's tree
    o, f, w = tracegen.random_paths(400, 30, 12, 2, seed=7)
    rng = np.random.default_rng(7)
    # distinct IDs spread over the whole uint64 range (an odd multiplier is a bijection mod 2^64)
    ids = rng.choice(10**9, size=400, replace=False).astype(np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    perm = rng.permutation(400)
    jo, jf, jw, unmatched = oracle.join_activity(o, f, ids, ids[perm], w[perm])
    assert unmatched == 0
    assert_tree_equal(oracle.build_tree(jo, jf, jw), oracle.build_tree(o, f, w), "self-registered")


def test_join_counts_unregistered_records_by_brute_force():
    o, f, w = tracegen.random_paths(50, 8, 6, 1, seed=3)
    rng = np.random.default_rng(3)
    ids = np.arange(50, dtype=np.uint64) * np.uint64(3)
    rec = rng.integers(0, 160, size=300).astype(np.uint64)
    rw = rng.integers(0, 2**64, size=(300, 1), dtype=np.uint64)
    jo, jf, jw, unmatched = oracle.join_activity(o, f, ids, rec, rw)
    registered = set(ids.tolist())
    assert unmatched == sum(1 for c in rec.tolist() if c not in registered)
    # brute force: the k-th matched record in order carries its registered path
    k = 0
    for r, c in enumerate(rec.tolist()):
        if c in registered:
            i = c // 3
            assert jf[jo[k]:jo[k + 1]].tolist() == f[o[i]:o[i + 1]].tolist()
            assert jw[k, 0] == rw[r, 0]
            k += 1
    assert k == jo.size - 1


def test_join_edge_cases():
    o, f, w, u = oracle.join_activity([0], [], [], [1, 2], [[1], [2]])
    assert (o.tolist(), f.size, w.shape, u) == ([0], 0, (0, 1), 2)
    o, f, w, u = oracle.join_activity([0, 2], [4, 4], [9], [], np.zeros((0, 3), np.uint64))
    assert (o.tolist(), f.size, w.shape, u) == ([0], 0, (0, 3), 0)


# ---- bottom-up view -----------------------------------------------------------------
# Events [1,2,1,2]:5, [2,3]:7, [9]:11, []:13.  By hand: excl(f) sums the events ending
# with f: 2 <- 5, 3 <- 7, 9 <- 11 (the empty path ends with no frame); incl(f) sums the
# events containing f once each: 1 <- 5, 2 <- 5 + 7, 3 <- 7, 9 <- 11 (frame 1 and 2 recur
# on the first path and count once).
def test_bottom_up_hand_worked():
    fr, ex, inc = oracle.bottom_up([0, 4, 6, 7, 7], [1, 2, 1, 2, 2, 3, 9], [[5], [7], [11], [13]])
    assert fr.tolist() == [1, 2, 3, 9]
    assert ex.ravel().tolist() == [0, 5, 7, 11]
    assert inc.ravel().tolist() == [5, 12, 7, 11]


def py_bottom_up_from_tree(t):
    """Second definition, from the tree: every node adds its exclusive sums to its frame;
    a node whose proper ancestors carry no node of its frame adds its inclusive sums
    (each event passes through exactly one such topmost node of each frame it contains)."""
    parent, frame = t["parent"], t["frame"]
    m = t["excl"].shape[1]
    mask = (1 << 64) - 1
    ex, inc = {}, {}
    for v in range(1, parent.size):
        f = int(frame[v])
        ex.setdefault(f, [0] * m)
        inc.setdefault(f, [0] * m)
        u, top = int(parent[v]), True
        while u != 0:
            if int(frame[u]) == f:
                top = False
                break
            u = int(parent[u])
        for j in range(m):
            ex[f][j] = (ex[f][j] + int(t["excl"][v, j])) & mask
            if top:
                inc[f][j] = (inc[f][j] + int(t["incl"][v, j])) & mask
    keys = sorted(ex)
    return keys, [ex[k] for k in keys], [inc[k] for k in keys]


@pytest.mark.parametrize("seed", range(6))
def test_bottom_up_events_match_the_tree_rule(seed):
    # small frame alphabets make recursion (repeated frames on a path) frequent
    o, f, w = tracegen.random_paths(300, 3 + seed, 12, 2, seed=seed)  # (events, frame ids, max length, M)
    fr, ex, inc = oracle.bottom_up(o, f, w)
    keys, tex, tinc = py_bottom_up_from_tree(oracle.build_tree(o, f, w))
    assert fr.tolist() == keys
    assert ex.tolist() == tex
    assert inc.tolist() == tinc


def test_bottom_up_closed_forms():
    # one path of distinct frames: every frame's incl is the path's weight
    fr, ex, inc = oracle.bottom_up([0, 5], [10, 20, 30, 40, 50], [[7]])
    assert fr.tolist() == [10, 20, 30, 40, 50]
    assert inc.ravel().tolist() == [7] * 5 and ex.ravel().tolist() == [0, 0, 0, 0, 7]
    # pure recursion of one frame: counted once in incl and once in excl
    fr, ex, inc = oracle.bottom_up([0, 4], [6, 6, 6, 6], [[9]])
    assert (fr.tolist(), ex.ravel().tolist(), inc.ravel().tolist()) == ([6], [9], [9])
    # the root's placeholder is no frame; an empty trace has an empty view
    fr, ex, inc = oracle.bottom_up([0, 0], [], [[3]])
    assert fr.size == 0 and ex.shape == (0, 1)


def test_bottom_up_exclusive_total():
    # every non-empty event ends with exactly one frame: the exclusive view sums to the total
    o, f, w = tracegen.random_paths(2000, 20, 50, 3, seed=9)
    fr, ex, inc = oracle.bottom_up(o, f, w)
    nonempty = np.diff(o) > 0
    assert np.array_equal(ex.sum(axis=0, dtype=np.uint64), w[nonempty].sum(axis=0, dtype=np.uint64))


# ---- ratio filters --------------------------------------------------------------------
# The hand-worked tree of the join pin: ids () (5) (5,7) (5,9) (5,9,2), inclusive
# 22 20 4 16 16; leaves are (5,7) and (5,9,2).  Above half of the root: 22/22, 20/22,
# 16/22, 16/22 -> nodes 0 1 3 4; among leaves only node 4 (4/22 is below).  A ratio equal
# to the threshold matches neither way: 11/22 against 1/2.
def test_filter_hand_worked():
    t = oracle.build_tree([0, 3, 5, 8, 8], [5, 9, 2, 5, 7, 5, 9, 2], [[10], [4], [6], [2]])
    assert oracle.filter_nodes(t, 0, +1, 1, 2, den="root").tolist() == [0, 1, 3, 4]
    assert oracle.filter_nodes(t, 0, +1, 1, 2, den="root", leaves_only=True).tolist() == [4]
    assert oracle.filter_nodes(t, 0, -1, 1, 2, den="root").tolist() == [2]
    assert oracle.filter_nodes(t, 0, +1, 16, 1).tolist() == [0, 1]        # incl > 16
    assert oracle.filter_nodes(t, 0, +1, 2, 1, num_excl=True).tolist() == [2, 4]  # excl > 2 (root's is 2)


def test_filter_matches_fractions():
    # an independent evaluation with fractions.Fraction for non-zero denominators, and
    # the cross-multiplied reading for zero ones (above: a > 0; below: never)
    from fractions import Fraction
    o, f, w = tracegen.random_paths(400, 15, 10, 3, seed=4)
    w[::7, 2] = 0  # zero denominators
    t = oracle.build_tree(o, f, w)
    parents = set(t["parent"][1:].tolist())
    for op in (+1, -1):
        for p, q in ((1, 3), (7, 2), (0, 1)):
            got = oracle.filter_nodes(t, 0, op, p, q, den="metric", den_metric=2).tolist()
            want = []
            for v in range(t["parent"].size):
                a, b = int(t["incl"][v, 0]), int(t["incl"][v, 2])
                if b == 0:
                    hit = op > 0 and a * q > 0
                else:
                    hit = Fraction(a, b) > Fraction(p, q) if op > 0 else Fraction(a, b) < Fraction(p, q)
                if hit:
                    want.append(v)
            assert got == want
    leaves = oracle.filter_nodes(t, 0, +1, 0, 1, leaves_only=True).tolist()
    assert leaves == [v for v in range(t["parent"].size) if v not in parents and int(t["incl"][v, 0]) > 0]


# ---- per-node statistics (count, minimum, sum of squares; mean and deviation) -------------
STAT_KEYS = ("count_excl", "count_incl", "min_excl", "min_incl", "sumsq_excl", "sumsq_incl")
U64_MAX = 2**64 - 1


def py_stats_brute(o, f, w):
    """Every prefix of every event as a node (ids: sorted prefixes, which is the
    canonical order), with the list of samples each node receives: excl from the events
    that end there, incl from the events that pass through it."""
    n, m = len(o) - 1, w.shape[1]
    paths = [tuple(int(x) for x in f[o[i]:o[i + 1]]) for i in range(n)]
    prefixes = sorted({p[:k] for p in paths for k in range(len(p) + 1)} | {()})
    ex = {p: [] for p in prefixes}
    inc = {p: [] for p in prefixes}
    for i, p in enumerate(paths):
        row = [int(x) for x in w[i]]
        ex[p].append(row)
        for k in range(len(p) + 1):
            inc[p[:k]].append(row)
    return prefixes, ex, inc, m


def assert_stats_match_brute(t, o, f, w):
    prefixes, ex, inc, m = py_stats_brute(o, f, w)
    assert t["parent"].size == len(prefixes)
    for v, p in enumerate(prefixes):
        for side, samples in (("excl", ex[p]), ("incl", inc[p])):
            assert int(t["count_" + side][v]) == len(samples)
            for j in range(m):
                xs = [r[j] for r in samples]
                assert int(t["min_" + side][v, j]) == (min(xs) if xs else U64_MAX)
                lo, hi = (int(x) for x in t["sumsq_" + side][v, j])
                assert lo | (hi << 64) == sum(x * x for x in xs) % 2**128


# Events (5,7) w=(3,1), (5) w=(5,2), () w=(4,0): nodes () (5) (5,7).  Metric 0 through the
# root: samples 3, 5, 4 -> count 3, min 3, sum of squares 50, mean 4, population deviation
# sqrt(2/3); through (5): 3, 5 -> mean 4, deviation 1; metric 1 through (5): 1, 2 -> mean
# 1.5, deviation 0.5.  Exclusive: one sample at each node, deviation 0.
def test_stats_hand_worked():
    t = oracle.build_tree([0, 2, 3, 3], [5, 7, 5], [[3, 1], [5, 2], [4, 0]], stats=True)
    assert t["count_excl"].tolist() == [1, 1, 1] and t["count_incl"].tolist() == [3, 2, 1]
    assert t["min_incl"].tolist() == [[3, 0], [3, 1], [3, 1]]
    assert t["min_excl"].tolist() == [[4, 0], [5, 2], [3, 1]]
    assert t["sumsq_incl"][:, :, 0].tolist() == [[50, 5], [34, 5], [9, 1]]
    assert not t["sumsq_incl"][:, :, 1].any()
    d = oracle.derived_stats(t)
    assert d["mean_incl"].tolist() == [[4.0, 1.0], [4.0, 1.5], [3.0, 1.0]]
    assert d["std_incl"][0, 0] == math.sqrt(2 / 3) and d["std_incl"][1].tolist() == [1.0, 0.5]
    assert not d["std_excl"].any()


@pytest.mark.parametrize("seed", range(6))
def test_stats_match_brute_force_and_statistics(seed):
    # small alphabets make paths share prefixes; values below 2^20 never wrap
    import statistics
    from fractions import Fraction
    o, f, w = tracegen.random_paths(120, 4 + seed, 6, 2, seed=300 + seed)
    w %= np.uint64(1 << 20)
    t = oracle.build_tree(o, f, w, stats=True)
    assert_stats_match_brute(t, o, f, w)
    prefixes, ex, inc, m = py_stats_brute(o, f, w)
    d = oracle.derived_stats(t)
    for v, p in enumerate(prefixes):
        for side, samples in (("excl", ex[p]), ("incl", inc[p])):
            for j in range(m):
                xs = [r[j] for r in samples]
                got_mean, got_std = d["mean_" + side][v, j], d["std_" + side][v, j]
                if not xs:
                    assert math.isnan(got_mean) and math.isnan(got_std)
                    continue
                assert got_mean == float(Fraction(sum(xs), len(xs)))
                want = statistics.pstdev(xs)
                assert abs(got_std - want) <= 2 * math.ulp(want)


def test_stats_wrap_and_extremes():
    # values near 2^64: squares wrap modulo 2^128, minima stay exact
    o, f, w = tracegen.random_paths(200, 5, 5, 2, seed=17)
    rng = np.random.default_rng(5)
    w = rng.integers(2**63, 2**64, size=w.shape, dtype=np.uint64)
    w[::11] = 0
    t = oracle.build_tree(o, f, w, stats=True)
    assert_stats_match_brute(t, o, f, w)


def test_stats_incremental_equals_one_shot():
    o, f, w = tracegen.random_paths(700, 20, 12, 3, seed=41)
    one = oracle.build_tree(o, f, w, stats=True)
    orc = oracle.Oracle(3, stats=True)
    for a, b in ((0, 250), (250, 251), (251, 700)):
        orc.ingest(*_subset(o, f, w, np.arange(a, b)))
    inc = orc.tree()
    orc.close()
    for k in STAT_KEYS + ("excl", "incl"):
        assert np.array_equal(one[k], inc[k]), k


@pytest.mark.parametrize("k", [1, 2, 7, 40])
def test_stats_closed_form_repeated_path(k):
    # one path of 4 frames taken k times with values 1..k: every node on it sees all k
    # samples (count k, min 1, mean (k+1)/2, deviation sqrt((k^2-1)/12)); only the end node
    # holds them exclusively
    o = np.arange(k + 1, dtype=np.int64) * 4
    f = np.tile(np.array([9, 3, 3, 1], np.uint32), k)
    w = np.arange(1, k + 1, dtype=np.uint64)[:, None]
    t = oracle.build_tree(o, f, w, stats=True)
    d = oracle.derived_stats(t)
    assert t["count_incl"].tolist() == [k] * 5 and t["count_excl"].tolist() == [0] * 4 + [k]
    assert t["min_incl"][:, 0].tolist() == [1] * 5 and t["min_excl"][:4, 0].tolist() == [U64_MAX] * 4
    assert int(t["sumsq_incl"][0, 0, 0]) == k * (k + 1) * (2 * k + 1) // 6
    assert d["mean_incl"][:, 0].tolist() == [(k + 1) / 2] * 5
    want = math.sqrt((k * k - 1) / 12)
    assert all(abs(x - want) <= 2 * math.ulp(max(want, 1e-300)) for x in d["std_incl"][:, 0])
    assert np.isnan(d["mean_excl"][:4]).all() and d["std_excl"][4, 0] == d["std_incl"][4, 0]


# The join of test_join_hand_worked with one event per call: ID 100 -> (5,7) once (4),
# ID 7 -> (5,9,2) twice (10 + 6), ID 3 -> () once (2), in registry order; 999 unmatched.
def test_join_per_call_hand_worked():
    o, f, w, unmatched = oracle.join_activity_calls([0, 2, 5, 5], [5, 7, 5, 9, 2], [100, 7, 3],
                                                    [7, 999, 100, 7, 3], [[10], [1], [4], [6], [2]])
    assert unmatched == 1 and o.tolist() == [0, 2, 5, 5] and f.tolist() == [5, 7, 5, 9, 2]
    assert w.ravel().tolist() == [4, 16, 2]
    t = oracle.build_tree(o, f, w, stats=True)
    assert t["incl"].ravel().tolist() == [22, 20, 4, 16, 16]  # the per-record tree's sums
    assert t["count_incl"].tolist() == [3, 2, 1, 1, 1] and t["min_incl"].ravel().tolist() == [2, 4, 4, 16, 16]


def test_join_per_call_and_per_record_give_one_sum_tree():
    o, f, w = tracegen.random_paths(300, 25, 10, 2, seed=23)
    rng = np.random.default_rng(23)
    ids = rng.permutation(10**6)[:300].astype(np.uint64)
    rec = np.concatenate([ids, ids[rng.integers(0, 300, 90)], np.arange(10**6, 10**6 + 20, dtype=np.uint64)])
    met = rng.integers(0, 2**64, size=(rec.size, 2), dtype=np.uint64)
    a = oracle.join_activity(o, f, ids, rec, met)
    b = oracle.join_activity_calls(o, f, ids, rec, met)
    assert a[3] == b[3] == 20 and b[0].size - 1 == 300
    ta, tb = oracle.build_tree(*a[:3]), oracle.build_tree(*b[:3])
    for k in ("parent", "frame", "depth", "excl", "incl"):
        assert np.array_equal(ta[k], tb[k]), k
