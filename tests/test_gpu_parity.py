"""GPU path vs the CPU oracle, element by element, through the C ABI (bit-exact:
every output is integer)."""
import os

import numpy as np
import pytest

import oracle
import tracegen
from conftest import load_golden
from gpu_util import assert_same, csr, gpu_tree, node_paths, to_dev, torch_or_skip

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    torch_or_skip()


@pytest.mark.parametrize("name", ["W1.txt", "W2.txt", "W3.txt", "W4.txt"])
def test_hand_worked(name):
    o, f, w, want = load_golden(name)
    assert_same(gpu_tree(o, f, w), want, name)


@pytest.mark.parametrize("seed", range(60))
def test_random_small_vs_brute(seed):
    o, f, w = tracegen.random_small(1 + (seed * 37) % 400, 2 + seed % 4, 8, 1 + seed % 3, seed)
    assert_same(gpu_tree(o, f, w), oracle.brute_tree(o, f, w) if o.size < 80 else oracle.build_tree(o, f, w),
                f"seed {seed}")


@pytest.mark.parametrize("seed", range(6))
def test_random_paths_many_tiles(seed):
    # thousands of events: many tiles, ragged last tile, several workgroups
    n = [1, 255, 257, 5000, 33333, 100_003][seed]
    o, f, w = tracegen.random_paths(n, 50 + seed * 100, 40, 1 + seed % 4, seed=100 + seed)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), f"n={n}")


def test_workload_tiny_full():
    o, f, w = tracegen.generate("tiny")
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), "tiny")


def test_workload_layered_1m_full():
    o, f, w = tracegen.generate("layered_1m")
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), "layered_1m")


@pytest.mark.parametrize("name,n", [("layered_16m", 1 << 18), ("deep_recursion", 1 << 16),
                                    ("merge_base", 1 << 17)])
def test_workload_scaled(name, n):
    o, f, w = tracegen.generate(name, n_events=n)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), f"{name}[{n}]")


# ---- edge cases ----------------------------------------------------------------------
def test_empty_input():
    t = gpu_tree(np.zeros(1, np.int64), np.zeros(0, np.uint32), np.zeros((0, 2), np.uint64))
    assert t["parent"].size == 1 and t["parent"][0] == 0xFFFFFFFF
    assert np.all(t["excl"] == 0) and np.all(t["incl"] == 0)


def test_only_zero_length_paths():
    o = np.zeros(6, np.int64)
    w = np.arange(1, 6, dtype=np.uint64).reshape(5, 1)
    t = gpu_tree(o, np.zeros(0, np.uint32), w)
    assert t["parent"].size == 1 and int(t["excl"][0, 0]) == 15 and int(t["incl"][0, 0]) == 15


def test_single_event_and_identical_events():
    o, f = csr([[5, 0xFFFFFFFF, 0, 7]])
    w = np.array([[42]], np.uint64)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), "single")
    o, f = csr([[9, 3, 3, 9, 0xFFFFFFFF]] * 5000)
    w = np.full((5000, 1), 3, np.uint64)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), "identical")


@pytest.mark.parametrize("L", [512, 6000, 20000])
def test_long_paths(L):
    # 6000 and 20000 frames exceed one tile's LDS staging: the workgroup-per-event path
    rng = np.random.default_rng(L)
    base = rng.integers(0, 2**32, size=L, dtype=np.uint64).astype(np.uint32)
    paths = [base.tolist(), base[: L // 2].tolist(), base.tolist(), (base[:-1].tolist() + [1]), [3, 4]]
    paths += [base[:k].tolist() for k in (1, 2, L - 1)]
    o, f = csr(paths)
    w = rng.integers(0, 2**64, size=(len(paths), 2), dtype=np.uint64)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), f"L={L}")


@pytest.mark.parametrize("shape", ["star", "star_with_empty", "comb"])
def test_one_node_per_path_windows(shape):
    # the emission takes 64 consecutive nodes per wave and finds their paths among the 64
    # paths from the one holding the first node: paths that add one node each (a star of
    # leaves under the root, or a comb of leaves hanging off one spine) put 64 paths in
    # every window, the most a window can hold; the empty path adds none
    rng = np.random.default_rng(12)
    if shape == "comb":
        spine = rng.integers(0, 2**32, size=700, dtype=np.uint64).astype(np.uint32).tolist()
        paths = [spine] + [spine[:k] + [0xFFFFFFF0 - k] for k in range(700)]
    else:
        paths = [[int(x)] for x in rng.permutation(5000)]
        if shape == "star_with_empty":
            paths += [[]] * 3
    order = rng.permutation(len(paths))
    o, f = csr([paths[i] for i in order])
    w = rng.integers(0, 2**64, size=(len(paths), 2), dtype=np.uint64)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), shape)


def test_mixed_long_and_short_in_one_tile():
    rng = np.random.default_rng(7)
    paths = [rng.integers(0, 5, size=rng.integers(0, 6)).tolist() for _ in range(300)]
    paths[17] = rng.integers(0, 5, size=9000).tolist()
    o, f = csr(paths)
    w = rng.integers(0, 1000, size=(300, 1), dtype=np.uint64)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), "mixed")


def test_wraparound_and_extreme_ids():
    o, f, w, want = load_golden("W3.txt")
    assert_same(gpu_tree(o, f, w), want)
    o, f = csr([[0xFFFFFFFF, 0], [0, 0xFFFFFFFF], [0x80000000], [0x7FFFFFFF, 0x80000000], []])
    w = np.array([[2**64 - 1], [2**63], [2**63], [5], [2**64 - 3]], np.uint64)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w))


def test_misaligned_frames_pointer():
    # frames view starting 1..3 elements into an allocation: unaligned 16-byte groups
    torch = torch_or_skip()
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.random_paths(3000, 30, 20, 2, seed=5)
    for shift in (1, 2, 3):
        to, tf, tw = to_dev(o, f, w)
        big = torch.zeros(tf.numel() + shift, dtype=torch.int32, device=tf.device)
        big[shift:] = tf
        tree = cct.build(to, big[shift:], tw)
        assert_same(tree.to_numpy(), oracle.build_tree(o, f, w), f"shift {shift}")
        tree.free()


# ---- forced conditions from the host ------------------------------------------------------
@pytest.mark.parametrize("bits", [0, 2, 5])
def test_forced_hash_collisions(monkeypatch, bits):
    monkeypatch.setenv("CCT_TEST_HASH_BITS", str(bits))
    o, f, w = tracegen.random_small(300, 4, 7, 2, seed=bits)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), f"bits={bits}")


@pytest.mark.parametrize("bits", [5, 9])
def test_forced_collisions_through_cache(monkeypatch, bits):
    # many events per distinct path, so workgroup caches hold paths whose hash and
    # length collide with others: a cached candidate that differs must not make an
    # event skip the slots before it on the probe sequence
    monkeypatch.setenv("CCT_TEST_HASH_BITS", str(bits))
    o, f, w = tracegen.random_small(20_000, 4, 7, 2, seed=40 + bits)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), f"bits={bits}")


@pytest.mark.parametrize("case", ["tiny", "layered_1m_part", "deep_part", "random_small", "random_paths", "long"])
def test_block_trie_order(monkeypatch, case):
    # the block-trie ranking must be usable (no fallback) and agree with the oracle and
    # with the comparison sort
    if case == "tiny":
        o, f, w = tracegen.generate("tiny")
    elif case == "layered_1m_part":
        o, f, w = tracegen.generate("layered_1m", n_events=200_000)
    elif case == "deep_part":
        o, f, w = tracegen.generate("deep_recursion", n_events=30_000)
    elif case == "random_small":
        o, f, w = tracegen.random_small(5000, 16, 9, 1, seed=77)
    elif case == "random_paths":
        o, f, w = tracegen.random_paths(20_000, 40, 70, 2, seed=78)
    else:  # paths of every length 0..300 over 3 frame ids: many full and partial blocks
        lens = np.arange(301)
        rng = np.random.default_rng(79)
        o = np.zeros(lens.size + 1, np.int64)
        o[1:] = np.cumsum(lens)
        f = rng.integers(0, 3, int(o[-1])).astype(np.uint32)
        w = rng.integers(0, 1000, (lens.size, 1)).astype(np.uint64)
    want = oracle.build_tree(o, f, w)
    monkeypatch.setenv("CCT_TEST_REQUIRE_TRIE", "1")
    assert_same(gpu_tree(o, f, w), want, f"{case} trie")
    monkeypatch.delenv("CCT_TEST_REQUIRE_TRIE")
    monkeypatch.setenv("CCT_TEST_MERGE_SORT", "1")
    assert_same(gpu_tree(o, f, w), want, f"{case} comparison sort")


@pytest.mark.parametrize("bits", [1, 4])
@pytest.mark.parametrize("sort", ["trie", "comparison"])
def test_forced_checkpoint_collisions(monkeypatch, bits, sort):
    # checkpoint hashes cut to a few bits: the fast orders (block trie, comparison sort,
    # the merge's gap search) meet colliding prefixes, their order is caught by the exact
    # check, and the exact comparison sort takes over; a build and two merges equal the
    # oracle
    import paper_2411_02797_amd as cct
    monkeypatch.setenv("CCT_TEST_CP_HASH_BITS", str(bits))
    if sort == "comparison":
        monkeypatch.setenv("CCT_TEST_MERGE_SORT", "1")
    o, f, w = tracegen.random_paths(4000, 3, 70, 2, seed=90 + bits)
    o2, f2, w2 = tracegen.random_paths(3000, 3, 90, 2, seed=95 + bits)
    o3, f3, w3 = tracegen.generate("deep_recursion", n_events=3000)
    w3 = np.repeat(w3, 2, axis=1)
    tree = cct.build(*to_dev(o, f, w))
    assert_same(tree.to_numpy(), oracle.build_tree(o, f, w), f"build bits={bits} {sort}")
    tree.merge(*to_dev(o2, f2, w2))
    tree.merge(*to_dev(o3, f3, w3))
    orc = oracle.Oracle(2)
    for t in ((o, f, w), (o2, f2, w2), (o3, f3, w3)):
        orc.ingest(*t)
    assert_same(tree.to_numpy(), orc.tree(), f"merges bits={bits} {sort}")
    orc.close()
    tree.free()


def test_forced_table_overflow_regrows(monkeypatch):
    monkeypatch.setenv("CCT_TEST_TABLE_CAP", "16")
    o, f, w = tracegen.random_paths(5000, 500, 12, 1, seed=9)
    assert_same(gpu_tree(o, f, w), oracle.build_tree(o, f, w), "regrow")


def test_exact_sort_mode_matches(monkeypatch):
    o, f, w = tracegen.generate("deep_recursion", n_events=20_000)
    want = oracle.build_tree(o, f, w)
    assert_same(gpu_tree(o, f, w), want, "checkpoint sort")
    monkeypatch.setenv("CCT_TEST_EXACT_SORT", "1")
    assert_same(gpu_tree(o, f, w), want, "exact sort")


# ---- algebraic laws ----------------------------------------------------------------------
def _subset(o, f, w, idx):
    lens = (o[1:] - o[:-1])[idx]
    oo = np.zeros(idx.size + 1, np.int64)
    oo[1:] = np.cumsum(lens)
    ff = np.concatenate([f[o[i]:o[i + 1]] for i in idx]) if idx.size else np.zeros(0, np.uint32)
    return oo, ff.astype(np.uint32), w[idx]


def test_permutation_invariance_and_determinism():
    o, f, w = tracegen.generate("layered_16m", n_events=50_000)
    a = gpu_tree(o, f, w)
    b = gpu_tree(o, f, w)
    for k in a:
        assert a[k].tobytes() == b[k].tobytes(), f"repeat differs in {k}"
    perm = np.random.default_rng(0).permutation(50_000)
    assert_same(gpu_tree(*_subset(o, f, w, perm)), a, "permuted")


def test_metrics_independent_columns():
    o, f, w = tracegen.random_paths(20_000, 300, 30, 4, seed=12)
    t = gpu_tree(o, f, w)
    for j in range(4):
        tj = gpu_tree(o, f, w[:, j:j + 1])
        assert np.array_equal(t["excl"].reshape(-1, 4)[:, j], tj["excl"].ravel())
        assert np.array_equal(t["incl"].reshape(-1, 4)[:, j], tj["incl"].ravel())


def test_merge_equals_one_shot():
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.generate("merge_base", n_events=40_000)
    chunks = [tracegen.generate("merge_chunk", n_events=10_000, chunk=c) for c in range(4)]
    tree = cct.build(*to_dev(o, f, w))
    orc = oracle.Oracle(4)
    orc.ingest(o, f, w)
    for (co, cf, cw) in chunks:
        tree.merge(*to_dev(co, cf, cw))
        orc.ingest(co, cf, cw)
        assert_same(tree.to_numpy(), orc.tree(), "incremental")
    # and equal to one GPU build over everything
    allo = np.concatenate([o[:-1]] + [c[0][:-1] + o[-1] + sum(x[0][-1] for x in chunks[:i])
                                      for i, c in enumerate(chunks)] + [[o[-1] + sum(x[0][-1] for x in chunks)]])
    allf = np.concatenate([f] + [c[1] for c in chunks])
    allw = np.concatenate([w] + [c[2] for c in chunks])
    assert_same(gpu_tree(allo, allf, allw), tree.to_numpy(), "one-shot")
    tree.free()


@pytest.mark.parametrize("full_sort", [False, True])
def test_merge_orders(monkeypatch, full_sort):
    # a merge keeps the previous order and merges this call's new paths into it (or,
    # forced, sorts every path again): merges that add no path, a few, and more new
    # paths than the tree holds
    import paper_2411_02797_amd as cct
    if full_sort:
        monkeypatch.setenv("CCT_TEST_FULL_SORT", "1")
    o, f, w = tracegen.generate("merge_base", n_events=20_000)
    tree = cct.build(*to_dev(o, f, w))
    orc = oracle.Oracle(4)
    orc.ingest(o, f, w)
    batches = [(o, f, w), tracegen.generate("merge_chunk", n_events=5_000, chunk=0),
               tracegen.random_paths(30_000, 5000, 40, 4, seed=21)]
    for k, b in enumerate(batches):
        tree.merge(*to_dev(*b))
        orc.ingest(*b)
        assert_same(tree.to_numpy(), orc.tree(), f"merge {k} (full sort {full_sort})")
    tree.free()
    orc.close()


def test_merge_into_empty_and_empty_merge():
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.random_paths(2000, 50, 10, 2, seed=3)
    tree = cct.build(*to_dev(np.zeros(1, np.int64), np.zeros(0, np.uint32), np.zeros((0, 2), np.uint64)))
    tree.merge(*to_dev(o, f, w))
    tree.merge(*to_dev(np.zeros(1, np.int64), np.zeros(0, np.uint32), np.zeros((0, 2), np.uint64)))
    assert_same(tree.to_numpy(), oracle.build_tree(o, f, w))
    tree.free()


# ---- queries ---------------------------------------------------------------------------------
@pytest.mark.parametrize("mode", ["index", "search", "collisions"])
def test_query_every_node_and_absent_paths(mode, monkeypatch):
    # the prefix index, the binary search, and the index with 3-bit keys (every lookup
    # meets many entries of other nodes with its key and must verify them)
    import paper_2411_02797_amd as cct
    torch = torch_or_skip()
    if mode == "search":
        monkeypatch.setenv("CCT_TEST_QUERY_SEARCH", "1")
    elif mode == "collisions":
        monkeypatch.setenv("CCT_TEST_QUERY_HASH_BITS", "3")
    o, f, w = tracegen.random_paths(3000, 40, 12, 2, seed=4)
    want = oracle.build_tree(o, f, w)
    tree = cct.build(*to_dev(o, f, w))
    U = want.n_nodes
    paths = node_paths(want, range(U))
    absent = [[123456789], paths[-1] + [987654321], [0xFFFFFFFF] * 3]
    qo, qf = csr(paths + absent)
    dev = torch.device("cuda", 0)
    ids, ex, inc = tree.query(torch.from_numpy(qo).to(dev), torch.from_numpy(qf.view(np.int32)).to(dev))
    ids = ids.cpu().numpy()
    assert np.array_equal(ids[:U], np.arange(U)) and np.all(ids[U:] == -1)
    assert np.array_equal(ex.cpu().numpy()[:U].view(np.uint64), want["excl"])
    assert np.array_equal(inc.cpu().numpy()[:U].view(np.uint64), want["incl"])
    assert np.all(inc.cpu().numpy()[U:] == 0)
    # the kept index follows a merge: the same queries against the merged tree
    o2, f2, w2 = tracegen.random_paths(2000, 60, 12, 2, seed=5)
    tree.merge(*to_dev(o2, f2, w2))
    oc = np.concatenate([o, o[-1] + o2[1:]])
    want2 = oracle.build_tree(oc, np.concatenate([f, f2]), np.concatenate([w, w2]))
    ids2, _, inc2 = tree.query(torch.from_numpy(qo).to(dev), torch.from_numpy(qf.view(np.int32)).to(dev))
    paths2 = node_paths(want2, range(want2.n_nodes))
    index_of = {tuple(p_): v for v, p_ in enumerate(paths2)}
    exp = np.array([index_of.get(tuple(p_), -1) for p_ in paths + absent])
    assert np.array_equal(ids2.cpu().numpy(), exp)
    hit = exp >= 0
    assert np.array_equal(inc2.cpu().numpy()[hit].view(np.uint64), want2["incl"][exp[hit]])
    tree.free()


@pytest.mark.parametrize("case", ["layered_1m_part", "random_paths"])
def test_one_stream_only(monkeypatch, case):
    # with no second stream (a test setting: the path taken when none can be created) the
    # aggregation, the fold and the sibling ordering all run on the caller's stream, in
    # order; the tree equals the oracle's, and a merge after it too
    if case == "layered_1m_part":
        o, f, w = tracegen.generate("layered_1m")
        n = 60000
        o, f, w = o[: n + 1].copy(), f[: o[n]].copy(), w[:n].copy()
    else:
        o, f, w = tracegen.random_paths(30000, 200, 40, 2, seed=91)
    ob, fb, wb = tracegen.random_paths(5000, 200, 40, w.shape[1], seed=92)
    monkeypatch.setenv("CCT_TEST_ONE_STREAM", "1")
    import paper_2411_02797_amd as cct
    tree = cct.build(*to_dev(o, f, w))
    assert_same(tree.to_numpy(), oracle.build_tree(o, f, w), case)
    tree.merge(*to_dev(ob, fb, wb))
    oc = np.concatenate([o, o[-1] + ob[1:]])
    want = oracle.build_tree(oc, np.concatenate([f, fb]), np.concatenate([w, wb]))
    assert_same(tree.to_numpy(), want, case + " merged")
    tree.free()


def test_concurrent_builds_on_two_threads():
    # distinct trees built and merged at the same time from two host threads, each on its
    # own stream: every call takes its own side stream, so neither waits for or corrupts
    # the other
    import threading

    import paper_2411_02797_amd as cct
    torch = torch_or_skip()
    results, errors = {}, []

    def work(k):
        try:
            st = torch.cuda.Stream()
            with torch.cuda.stream(st):
                o, f, w = tracegen.random_paths(20000, 300 + 50 * k, 30, 2, seed=70 + k)
                o2, f2, w2 = tracegen.random_paths(8000, 300 + 50 * k, 30, 2, seed=80 + k)
                for _ in range(3):
                    tree = cct.build(*to_dev(o, f, w), stats=True)
                    tree.merge(*to_dev(o2, f2, w2))
                    got = tree.to_numpy()
                    tree.free()
            oc = np.concatenate([o, o[-1] + o2[1:]])
            results[k] = (got, oracle.build_tree(oc, np.concatenate([f, f2]), np.concatenate([w, w2])))
        except Exception as e:  # reported by the main thread
            errors.append(repr(e))

    threads = [threading.Thread(target=work, args=(k,)) for k in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for k, (got, want) in results.items():
        assert_same(got, want, f"thread {k}")
