"""cct_merge_activity (correlation-ID join of an activity flush, then merge) against the
oracle: the oracle joins by its definition (a dictionary from ID to registered path, one
event per matched record) and ingests the joined batch into the same trie as the base
trace.  Every output array is compared element by element, bit-exact, and the count of
unmatched records must agree."""
import numpy as np
import pytest

import oracle
import tracegen
from gpu_util import assert_same, to_dev, torch_or_skip

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    torch_or_skip()


def _u64(a):
    torch = torch_or_skip()
    a = np.ascontiguousarray(a, np.uint64)
    return torch.from_numpy(a.view(np.int64)).to(torch.device("cuda", 0))


def flush(n_reg, n_rec, m, seed, unregistered=0.2, max_len=40, n_frames=12, repeat=0.3):
    """A registry of n_reg paths under distinct IDs spread over uint64 (0 and 2^64 - 1
    among them) and n_rec records: a share name unregistered IDs, and registered IDs
    repeat (several records per launch)."""
    ro, rf, _ = tracegen.random_paths(n_reg, max_len, n_frames, 1, seed=seed)
    rng = np.random.default_rng(seed)
    ids = rng.choice(10**12, size=n_reg, replace=False).astype(np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    ids[0] = np.uint64(0)
    if n_reg > 1:
        ids[1] = np.uint64(2**64 - 1)
    hot = rng.choice(n_reg, size=max(1, n_reg // 20))  # a few launches with many records
    pick = np.where(rng.random(n_rec) < repeat, rng.choice(hot, size=n_rec), rng.integers(0, n_reg, size=n_rec))
    rec = ids[pick].copy()
    unreg = rng.random(n_rec) < unregistered
    fresh = (rng.integers(0, 2**63, size=n_rec, dtype=np.int64).astype(np.uint64) << np.uint64(1)) | np.uint64(1)
    rec[unreg] = fresh[unreg]
    w = rng.integers(0, 2**64, size=(n_rec, m), dtype=np.uint64)
    return ro, rf, ids, rec, w


def run_case(base, reg, m):
    import paper_2411_02797_amd as cct
    o, f, w = base
    ro, rf, ids, rec, rw = reg
    tree = cct.build(*to_dev(o, f, w))
    to, tf, _ = to_dev(ro, rf, np.zeros((ro.size - 1, 1), np.uint64))
    unmatched = tree.merge_activity(to, tf, _u64(ids), _u64(rec), _u64(rw.reshape(-1, m)))
    got = tree.to_numpy()
    tree.free()
    jo, jf, jw, want_unmatched = oracle.join_activity(ro, rf, ids, rec, rw)
    orc = oracle.Oracle(m)
    orc.ingest(o, f, w)
    orc.ingest(jo, jf, jw)
    want = orc.tree()
    orc.close()
    assert unmatched == want_unmatched
    return got, want


@pytest.mark.parametrize("seed,m", [(1, 1), (2, 3), (3, 8)])
def test_join_then_merge(seed, m):
    base = tracegen.random_paths(3000, 40, 12, m, seed=100 + seed)
    reg = flush(2500, 4000, m, seed)
    got, want = run_case(base, reg, m)
    assert_same(got, want, f"seed {seed} M {m}")


def test_join_into_an_empty_tree():
    m = 2
    base = (np.zeros(1, np.int64), np.zeros(0, np.uint32), np.zeros((0, m), np.uint64))
    reg = flush(700, 1200, m, 9, unregistered=0.0)
    got, want = run_case(base, reg, m)
    assert_same(got, want, "empty tree")


def test_join_larger_flush():
    # a DL-shaped flush: registered paths from the layered program (long shared prefixes),
    # one record per launch in shuffled order plus repeats, 5% unregistered
    m = 4
    co, cf, _ = tracegen.generate("merge_chunk", chunk=0)
    n = 200_000
    ro = co[:n + 1].copy()
    rf = cf[:ro[-1]].copy()
    rng = np.random.default_rng(11)
    ids = rng.permutation(n).astype(np.uint64) + np.uint64(1 << 40)
    rec = np.concatenate([ids[rng.permutation(n)], ids[rng.integers(0, n, size=n // 4)]])
    unreg = rng.random(rec.size) < 0.05
    rec[unreg] = rng.integers(0, 1 << 39, size=int(unreg.sum())).astype(np.uint64)
    rw = rng.integers(0, 2**40, size=(rec.size, m), dtype=np.uint64)
    base = tracegen.random_paths(5000, 60, 200, m, seed=5)
    got, want = run_case(base, (ro, rf, ids, rec, rw), m)
    assert_same(got, want, "200k registered paths, 250k records")


def test_all_records_unmatched_leave_the_tree_unchanged():
    import paper_2411_02797_amd as cct
    m = 1
    o, f, w = tracegen.random_paths(800, 20, 8, m, seed=4)
    tree = cct.build(*to_dev(o, f, w))
    before = tree.to_numpy()
    ro, rf, ids, _, _ = flush(300, 10, m, 4)
    registered = set(ids.tolist())
    rec = np.array([c for c in range(2, 1002, 2) if c not in registered], np.uint64)
    to, tf, _ = to_dev(ro, rf, np.zeros((ro.size - 1, 1), np.uint64))
    un = tree.merge_activity(to, tf, _u64(ids), _u64(rec), _u64(np.ones((rec.size, m), np.uint64)))
    assert un == rec.size
    assert_same(tree.to_numpy(), before, "all unmatched")
    # no records, and an empty registry
    assert tree.merge_activity(to, tf, _u64(ids), _u64(np.zeros(0, np.uint64)), _u64(np.zeros((0, m), np.uint64))) == 0
    eo, ef, _ = to_dev(np.zeros(1, np.int64), np.zeros(0, np.uint32), np.zeros((0, 1), np.uint64))
    assert tree.merge_activity(eo, ef, _u64(np.zeros(0, np.uint64)), _u64(rec), _u64(np.ones((rec.size, m), np.uint64))) \
        == rec.size
    assert_same(tree.to_numpy(), before, "no records / empty registry")
    tree.free()


def _status(fn):
    import paper_2411_02797_amd as cct
    with pytest.raises(cct.CctError) as ei:
        fn()
    return ei.value.name


def test_errors_leave_the_tree_unchanged():
    import paper_2411_02797_amd as cct
    m = 2
    o, f, w = tracegen.random_paths(1000, 30, 10, m, seed=6)
    tree = cct.build(*to_dev(o, f, w))
    before = tree.to_numpy()
    ro, rf, ids, rec, rw = flush(400, 600, m, 6)
    to, tf, _ = to_dev(ro, rf, np.zeros((ro.size - 1, 1), np.uint64))
    # a repeated registered ID (far apart in the registry)
    rep = ids.copy()
    rep[350] = rep[17]
    assert _status(lambda: tree.merge_activity(to, tf, _u64(rep), _u64(rec), _u64(rw))) == "CCT_EINVAL"
    # malformed registry offsets
    bad = to.clone()
    bad[200] = bad[199] - 1
    assert _status(lambda: tree.merge_activity(bad, tf, _u64(ids), _u64(rec), _u64(rw))) == "CCT_EINVAL"
    # metric count differs from the tree's
    assert _status(lambda: tree.merge_activity(to, tf, _u64(ids), _u64(rec), _u64(np.zeros((rec.size, 3), np.uint64)))) \
        == "CCT_EMISMATCH"
    assert_same(tree.to_numpy(), before, "after failed calls")
    # still usable
    tree.merge_activity(to, tf, _u64(ids), _u64(rec), _u64(rw))
    jo, jf, jw, _ = oracle.join_activity(ro, rf, ids, rec, rw)
    orc = oracle.Oracle(m)
    orc.ingest(o, f, w)
    orc.ingest(jo, jf, jw)
    assert_same(tree.to_numpy(), orc.tree(), "merge after failures")
    orc.close()
    tree.free()


@pytest.mark.parametrize("k", [1, 3, 6, 9, 12, 15, 20, 30])
def test_allocation_failure(monkeypatch, k):
    import paper_2411_02797_amd as cct
    m = 1
    o, f, w = tracegen.random_paths(1500, 30, 10, m, seed=k)
    tree = cct.build(*to_dev(o, f, w))
    before = tree.to_numpy()
    ro, rf, ids, rec, rw = flush(500, 900, m, 50 + k)
    to, tf, _ = to_dev(ro, rf, np.zeros((ro.size - 1, 1), np.uint64))
    args = (to, tf, _u64(ids), _u64(rec), _u64(rw))
    monkeypatch.setenv("CCT_TEST_FAIL_ALLOC", str(k))
    try:
        tree.merge_activity(*args)
        merged = True
    except cct.CctError as e:
        assert e.name == "CCT_ENOMEM"
        merged = False
    monkeypatch.delenv("CCT_TEST_FAIL_ALLOC")
    if not merged:
        assert_same(tree.to_numpy(), before, "unchanged after ENOMEM")
        tree.merge_activity(*args)
    jo, jf, jw, _ = oracle.join_activity(ro, rf, ids, rec, rw)
    orc = oracle.Oracle(m)
    orc.ingest(o, f, w)
    orc.ingest(jo, jf, jw)
    assert_same(tree.to_numpy(), orc.tree(), "merged")
    orc.close()
    tree.free()


@pytest.mark.parametrize("seed", [21, 22])
def test_dense_ids_with_holes(seed):
    # registered IDs: a random 70% of a counter range (the direct table is used, with
    # holes); records name registered IDs, holes, and IDs just below and above the range
    m = 2
    ro, rf, _ = tracegen.random_paths(3000, 35, 14, 1, seed=seed)
    rng = np.random.default_rng(seed)
    base = np.uint64(2**63 - 1000)
    pool = np.arange(4300, dtype=np.uint64) + base
    ids = rng.permutation(rng.choice(pool, size=3000, replace=False))
    holes = np.setdiff1d(pool, ids)
    rec = np.concatenate([ids[rng.integers(0, 3000, 5000)], holes[:200], base - np.arange(1, 50, dtype=np.uint64),
                          base + np.uint64(4300) + np.arange(50, dtype=np.uint64)])
    rec = rec[rng.permutation(rec.size)]
    rw = rng.integers(0, 2**64, size=(rec.size, m), dtype=np.uint64)
    other = tracegen.random_paths(2000, 35, 14, m, seed=seed + 1)
    got, want = run_case(other, (ro, rf, ids, rec, rw), m)
    assert_same(got, want, f"dense IDs, seed {seed}")
    # a repeated ID inside the dense range is rejected
    import paper_2411_02797_amd as cct
    tree = cct.build(*to_dev(*other))
    rep = ids.copy()
    rep[2999] = rep[5]
    to, tf, _ = to_dev(ro, rf, np.zeros((ro.size - 1, 1), np.uint64))
    assert _status(lambda: tree.merge_activity(to, tf, _u64(rep), _u64(rec), _u64(rw))) == "CCT_EINVAL"
    tree.free()
