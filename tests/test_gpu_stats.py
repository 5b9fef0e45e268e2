"""cct_build_stats / cct_stats (per-node count, minimum, sum of squares, mean and
population deviation) against the oracle tree built with statistics from the same
events: the integer arrays bit-exact, the float64 mean and deviation within 4 units in the
last place of the oracle's exactly rounded values (the kernel rounds at most three times:
the 192-bit integer to float64, the square root and the division), NaN in the same
places."""
import ctypes

import numpy as np
import pytest

import oracle
import tracegen
from gpu_util import to_dev, torch_or_skip

pytestmark = pytest.mark.gpu

INT_FIELDS = ("count_excl", "count_incl", "min_excl", "min_incl", "sumsq_excl", "sumsq_incl")


@pytest.fixture(autouse=True)
def _gpu():
    torch_or_skip()


def gpu_stats(tree):
    out = tree.stats(device="cpu")
    return {k: (v.numpy().view(np.uint64) if v.dtype.is_floating_point is False else v.numpy()) for k, v in out.items()}


def assert_close_ulp(got, want, ctx):
    gn, wn = np.isnan(got), np.isnan(want)
    assert np.array_equal(gn, wn), f"{ctx}: NaN at {np.flatnonzero((gn != wn).ravel())[:8]}"
    g, w = got[~wn], want[~wn]
    bad = np.abs(g - w) > 4 * np.spacing(np.abs(w))
    assert not bad.any(), f"{ctx}: {bad.sum()} values off, e.g. {g[bad][:3]} vs {w[bad][:3]}"


def assert_stats(got, want_tree, ctx, nodes=None):
    for k in INT_FIELDS:
        g, w = got[k], want_tree[k]
        if nodes is not None:
            g = g[nodes]
            w = w[nodes]
        if not np.array_equal(g, w):
            bad = np.flatnonzero((g != w).reshape(g.shape[0], -1).any(axis=1))
            raise AssertionError(f"{ctx}: {k} differs at nodes {bad[:8]} (of {bad.size})")
    want = oracle.derived_stats(want_tree, nodes)
    for k, w in want.items():
        g = got[k] if nodes is None else got[k][nodes]
        assert_close_ulp(g, w, f"{ctx}: {k}")


def check_tree(tree, want_tree, ctx):
    arrs = tree.to_numpy()
    for k in ("parent", "frame", "depth", "excl", "incl"):
        assert np.array_equal(arrs[k], want_tree[k]), f"{ctx}: {k}"
    assert_stats(gpu_stats(tree), want_tree, ctx)


@pytest.mark.parametrize("seed,n_ids,m", [(1, 6, 1), (2, 40, 2), (3, 300, 3), (4, 3000, 8)])
def test_stats_match_oracle(seed, n_ids, m):
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.random_paths(8000, n_ids, 30, m, seed=seed)
    w %= np.uint64(1 << 40)
    tree = cct.build(*to_dev(o, f, w), stats=True)
    check_tree(tree, oracle.build_tree(o, f, w, stats=True), f"seed {seed}")
    tree.free()


def test_stats_full_range_values():
    # squares wrap modulo 2^128 and sums modulo 2^64; n*S2 - S1^2 can turn negative (NaN)
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.random_paths(5000, 30, 12, 2, seed=9)
    rng = np.random.default_rng(9)
    w = rng.integers(0, 2**64, size=w.shape, dtype=np.uint64)
    w[::5, 1] = np.uint64(2**64 - 1)
    w[::7, 0] = 0
    tree = cct.build(*to_dev(o, f, w), stats=True)
    check_tree(tree, oracle.build_tree(o, f, w, stats=True), "full range")
    tree.free()


MODES = pytest.mark.parametrize("atomic", [False, True], ids=["staged", "atomic"])


@MODES
def test_stats_hot_and_cold_paths(atomic, monkeypatch):
    # one path takes most events (LDS maps, same-address atomics); 150,000 distinct paths
    # overflow every workgroup's map (staged lists, or device atomics when forced)
    import paper_2411_02797_amd as cct
    if atomic:
        monkeypatch.setenv("CCT_TEST_STATS_ATOMIC", "1")
    n = 200_000
    rng = np.random.default_rng(12)
    hot = rng.random(n) < 0.6
    lens = np.where(hot, 5, rng.integers(1, 9, n))
    o = np.zeros(n + 1, np.int64)
    np.cumsum(lens, out=o[1:])
    f = rng.integers(0, 1 << 20, o[-1], dtype=np.uint32)
    for i in np.flatnonzero(hot)[:]:
        f[o[i]:o[i + 1]] = [1, 2, 3, 4, 5]
    w = rng.integers(0, 1 << 30, size=(n, 2), dtype=np.uint64)
    tree = cct.build(*to_dev(o, f, w), stats=True)
    check_tree(tree, oracle.build_tree(o, f, w, stats=True), "hot and cold")
    tree.free()


@MODES
def test_stats_follow_merges(atomic, monkeypatch):
    # a base, a merge of mostly known paths, and one with more new paths than the tree
    # holds (the path arrays grow)
    import paper_2411_02797_amd as cct
    if atomic:
        monkeypatch.setenv("CCT_TEST_STATS_ATOMIC", "1")
    m = 3
    batches = [tracegen.random_paths(3000, 20, 10, m, seed=30),
               tracegen.random_paths(2000, 20, 10, m, seed=31),
               tracegen.random_paths(9000, 400, 25, m, seed=32)]
    orc = oracle.Oracle(m, stats=True)
    tree = None
    for k, (o, f, w) in enumerate(batches):
        w %= np.uint64(1 << 32)
        if tree is None:
            tree = cct.build(*to_dev(o, f, w), stats=True)
        else:
            tree.merge(*to_dev(o, f, w))
        orc.ingest(o, f, w)
        check_tree(tree, orc.tree(), f"after batch {k}")
    orc.close()
    tree.free()


def test_stats_with_table_regrow(monkeypatch):
    import paper_2411_02797_amd as cct
    monkeypatch.setenv("CCT_TEST_TABLE_CAP", "64")
    o, f, w = tracegen.random_paths(6000, 200, 12, 2, seed=33)
    tree = cct.build(*to_dev(o, f, w), stats=True)
    o2, f2, w2 = tracegen.random_paths(4000, 300, 12, 2, seed=34)
    tree.merge(*to_dev(o2, f2, w2))
    oc = np.concatenate([o, o[-1] + o2[1:]])
    check_tree(tree, oracle.build_tree(oc, np.concatenate([f, f2]), np.concatenate([w, w2]), stats=True), "regrow")
    tree.free()


@MODES
def test_stats_of_activity_flushes(atomic, monkeypatch):
    # one sample per registered call with records (the sum of its records)
    import paper_2411_02797_amd as cct
    if atomic:
        monkeypatch.setenv("CCT_TEST_STATS_ATOMIC", "1")
    torch = torch_or_skip()
    m = 2
    o, f, w = tracegen.random_paths(2000, 25, 10, m, seed=40)
    tree = cct.build(*to_dev(o, f, w), stats=True)
    orc = oracle.Oracle(m, stats=True)
    orc.ingest(o, f, w)
    rng = np.random.default_rng(40)
    for flush in range(2):
        ro, rf, _ = tracegen.random_paths(3000, 25, 10, m, seed=41 + flush)
        ids = (rng.permutation(10**7)[:3000] + 10**7 * flush).astype(np.uint64)
        rec = np.concatenate([ids[:2500], ids[rng.integers(0, 2500, 400)], np.uint64(5 * 10**7) + np.arange(30, dtype=np.uint64)])
        rng.shuffle(rec)
        met = rng.integers(0, 1 << 30, size=(rec.size, m), dtype=np.uint64)
        dev = torch.device("cuda", 0)
        tree.merge_activity(*to_dev(ro, rf, np.zeros((3000, m), np.uint64))[:2],
                            torch.from_numpy(ids.view(np.int64)).to(dev),
                            torch.from_numpy(rec.view(np.int64)).to(dev), torch.from_numpy(met.view(np.int64)).to(dev))
        bo, bf, bw, _ = oracle.join_activity_calls(ro, rf, ids, rec, met)
        orc.ingest(bo, bf, bw)
        check_tree(tree, orc.tree(), f"flush {flush}")
    orc.close()
    tree.free()


def test_stats_edge_trees():
    import paper_2411_02797_amd as cct
    # no events; only empty paths; one path
    cases = [(np.zeros(1, np.int64), np.zeros(0, np.uint32), np.zeros((0, 2), np.uint64)),
             (np.zeros(4, np.int64), np.zeros(0, np.uint32), np.array([[3, 1], [5, 0], [4, 9]], np.uint64)),
             (np.array([0, 3], np.int64), np.array([7, 7, 7], np.uint32), np.array([[2**64 - 1, 0]], np.uint64))]
    for k, (o, f, w) in enumerate(cases):
        tree = cct.build(*to_dev(o, f, w), stats=True)
        check_tree(tree, oracle.build_tree(o, f, w, stats=True), f"case {k}")
        tree.free()


def test_stats_fields_and_errors():
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.random_paths(1000, 20, 8, 2, seed=50)
    tree = cct.build(*to_dev(o, f, w), stats=True)
    want = oracle.build_tree(o, f, w, stats=True)
    part = tree.stats(device="cpu", fields=("min_incl", "std_excl"))
    assert set(part) == {"min_incl", "std_excl"}
    assert np.array_equal(part["min_incl"].numpy().view(np.uint64), want["min_incl"])
    tree.free()
    plain = cct.build(*to_dev(o, f, w))
    with pytest.raises(cct.CctError):
        plain.stats()
    lib = cct.load_library()
    assert lib.cct_stats(plain.handle, None, None) == -1
    plain.free()


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_stats_full_size():
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.generate("layered_16m")
    print(f"layered_16m: N={o.size - 1:,}: building with statistics", flush=True)
    tree = cct.build(*to_dev(o, f, w), stats=True)
    got = gpu_stats(tree)
    tree.free()
    cct.release_cached_memory()
    print("layered_16m: oracle", flush=True)
    want = oracle.build_tree(o, f, w, stats=True)
    print("layered_16m: oracle done", flush=True)
    nodes = np.random.default_rng(1).choice(want["parent"].size, 20_000, replace=False)
    nodes = np.unique(np.concatenate([nodes, [0, 1, want["parent"].size - 1]]))
    for k in INT_FIELDS:
        assert np.array_equal(got[k], want[k]), k
    assert_stats(got, want, "layered_16m", nodes)
