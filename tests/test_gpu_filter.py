"""cct_filter (ratio tests over the tree's nodes) against the oracle's exact-integer
filter on the same tree: the lists of matching node ids must be equal."""
import ctypes
import itertools

import numpy as np
import pytest

import oracle
import tracegen
from gpu_util import to_dev, torch_or_skip

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    torch_or_skip()


def tree_pair(seed, full_range):
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.random_paths(5000, 12, 25, 3, seed=seed)
    if full_range:  # sums near 2^64: the 128-bit products carry into the high word
        rng = np.random.default_rng(seed)
        w = rng.integers(0, 2**64, size=w.shape, dtype=np.uint64)
    w[::9, 2] = 0  # zero denominators on some nodes
    tree = cct.build(*to_dev(o, f, w))
    return tree, oracle.build_tree(o, f, w)


THRESHOLDS = [(0, 1), (1, 1), (1, 1000), (3, 7), (2**63, 3), (2**64 - 1, 1), (1, 2**64 - 1)]


@pytest.mark.parametrize("seed,full_range", [(1, False), (2, True)])
def test_filters_match_oracle(seed, full_range):
    tree, want_tree = tree_pair(seed, full_range)
    for (p, q), op, den, num_excl, den_excl, leaves in itertools.product(
            THRESHOLDS, (+1, -1), ("one", "metric", "root"), (False, True), (False, True), (False, True)):
        if den != "metric" and den_excl:
            continue
        kw = dict(num_excl=num_excl, den=den, den_metric=2 if den == "metric" else 0, den_excl=den_excl,
                  leaves_only=leaves)
        got = tree.filter(0, op, p, q, **kw).cpu().numpy()
        want = oracle.filter_nodes(want_tree, 0, op, p, q, **kw)
        assert np.array_equal(got, want), f"threshold {p}/{q} op {op} {kw}: {got.size} vs {want.size} matches"
    tree.free()


def test_presets():
    tree, want_tree = tree_pair(3, False)
    assert np.array_equal(tree.hotspots(0, 1, 50).cpu().numpy(),
                          oracle.filter_nodes(want_tree, 0, +1, 1, 50, den="root", leaves_only=True))
    assert np.array_equal(tree.small_kernels(0, 1, 5, 1).cpu().numpy(),
                          oracle.filter_nodes(want_tree, 0, -1, 5, 1, den="metric", den_metric=1))
    assert np.array_equal(tree.cpu_latency(2, 0, 1, 4).cpu().numpy(),
                          oracle.filter_nodes(want_tree, 2, +1, 1, 4, den="metric", den_metric=0))
    tree.free()


def test_capacity_and_errors():
    import paper_2411_02797_amd as cct
    torch = torch_or_skip()
    tree, want_tree = tree_pair(4, False)
    lib = cct.load_library()
    want = oracle.filter_nodes(want_tree, 0, +1, 1, 1)  # incl > 1
    k = ctypes.c_int64(-1)
    out = torch.full((7,), -5, dtype=torch.int64, device="cuda")
    spec = cct._FilterSpec(0, 0, 0, 0, 0, 1, 1, 1, 0)
    assert lib.cct_filter(tree.handle, ctypes.byref(spec), None, 5, ctypes.c_void_p(out.data_ptr()), ctypes.byref(k)) == 0
    assert k.value == want.size > 5
    assert out.cpu().tolist() == want[:5].tolist() + [-5, -5]
    for bad in (cct._FilterSpec(3, 0, 0, 0, 0, 1, 1, 1, 0), cct._FilterSpec(0, 0, 1, 9, 0, 1, 1, 1, 0),
                cct._FilterSpec(0, 0, 3, 0, 0, 1, 1, 1, 0), cct._FilterSpec(0, 0, 0, 0, 0, 0, 1, 1, 0),
                cct._FilterSpec(0, 0, 0, 0, 0, 1, 1, 0, 0)):
        assert lib.cct_filter(tree.handle, ctypes.byref(bad), None, 0, None, ctypes.byref(k)) == -1  # CCT_EINVAL
    tree.free()


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_filters_full_size():
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.generate("layered_16m")
    tree = cct.build(*to_dev(o, f, w))
    root = tree.to_numpy()["incl"][0]
    p, q = int(root[0]), int(root[1])  # threshold only: the root's ratio of metric 0 to metric 1
    got = [tree.hotspots(0, 1, 1000).cpu().numpy(),
           tree.filter(0, -1, p, q, den="metric", den_metric=1).cpu().numpy()]
    tree.free()
    cct.release_cached_memory()
    print(f"layered_16m: {got[0].size} hotspots, {got[1].size} nodes below the root's ratio; oracle", flush=True)
    want_tree = oracle.build_tree(o, f, w)
    assert int(want_tree["incl"][0, 0]) == p and int(want_tree["incl"][0, 1]) == q
    print("layered_16m: oracle tree done", flush=True)
    assert np.array_equal(got[0], oracle.filter_nodes(want_tree, 0, +1, 1, 1000, den="root", leaves_only=True))
    assert np.array_equal(got[1], oracle.filter_nodes(want_tree, 0, -1, p, q, den="metric", den_metric=1))
