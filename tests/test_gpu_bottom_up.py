"""cct_bottom_up (the bottom-up view) against the oracle's view computed from the events:
frames, exclusive and inclusive sums compared element by element, bit-exact."""
import ctypes

import numpy as np
import pytest

import oracle
import tracegen
from gpu_util import to_dev, torch_or_skip

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    torch_or_skip()


def gpu_view(tree):
    v = tree.bottom_up(device="cpu")
    return (v["frames"].numpy().view(np.uint32), v["excl"].numpy().view(np.uint64),
            v["incl"].numpy().view(np.uint64))


def assert_view(got, want, ctx):
    for name, g, w in zip(("frames", "excl", "incl"), got, want):
        assert g.shape == w.shape, f"{ctx}: {name} shape {g.shape} vs {w.shape}"
        if not np.array_equal(g, w):
            bad = np.flatnonzero((g != w).ravel())
            raise AssertionError(f"{ctx}: {name} differs at {bad[:8]} (of {bad.size})")


@pytest.mark.parametrize("seed,n_frames,m", [(1, 3, 1), (2, 6, 2), (3, 40, 8), (4, 2000, 3)])
def test_view_matches_oracle(seed, n_frames, m):
    # small alphabets: frames recur on a path (recursion); large: mostly distinct
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.random_paths(6000, n_frames, 40, m, seed=seed)  # (events, frame ids, max length, M)
    tree = cct.build(*to_dev(o, f, w))
    got = gpu_view(tree)
    tree.free()
    assert_view(got, oracle.bottom_up(o, f, w), f"seed {seed}")


def test_view_unsigned_frame_order_and_high_ids():
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.random_paths(3000, 25, 30, 2, seed=8)
    f = (f.astype(np.uint64) * np.uint64(0x9E3779B1) % np.uint64(2**32)).astype(np.uint32)  # ids over all of uint32
    tree = cct.build(*to_dev(o, f, w))
    got = gpu_view(tree)
    tree.free()
    assert np.all(np.diff(got[0].astype(np.int64)) > 0)
    assert_view(got, oracle.bottom_up(o, f, w), "high ids")


def test_view_follows_merges():
    import paper_2411_02797_amd as cct
    m = 2
    o, f, w = tracegen.random_paths(4000, 30, 8, m, seed=10)
    tree = cct.build(*to_dev(o, f, w))
    assert_view(gpu_view(tree), oracle.bottom_up(o, f, w), "before merge")
    assert_view(gpu_view(tree), oracle.bottom_up(o, f, w), "kept view")
    o2, f2, w2 = tracegen.random_paths(3000, 30, 12, m, seed=11)
    tree.merge(*to_dev(o2, f2, w2))
    oc = np.concatenate([o, o[-1] + o2[1:]])
    assert_view(gpu_view(tree), oracle.bottom_up(oc, np.concatenate([f, f2]), np.concatenate([w, w2])), "after merge")
    tree.free()


def test_view_of_trees_without_frames():
    import paper_2411_02797_amd as cct
    for o in (np.zeros(1, np.int64), np.zeros(5, np.int64)):  # no events; four empty paths
        n = o.size - 1
        tree = cct.build(*to_dev(o, np.zeros(0, np.uint32), np.ones((n, 2), np.uint64)))
        fr, ex, inc = gpu_view(tree)
        tree.free()
        assert fr.size == 0 and ex.shape == (0, 2) and inc.shape == (0, 2)


def test_capacity_protocol():
    # capacity below K: nothing is written, K is returned; then a full copy
    import paper_2411_02797_amd as cct
    torch = torch_or_skip()
    o, f, w = tracegen.random_paths(1000, 20, 15, 1, seed=12)
    tree = cct.build(*to_dev(o, f, w))
    lib = cct.load_library()
    k = ctypes.c_int64(-1)
    dev = torch.device("cuda", 0)
    fr = torch.full((4,), -7, dtype=torch.int32, device=dev)
    assert lib.cct_bottom_up(tree.handle, None, 4, ctypes.c_void_p(fr.data_ptr()), None, None, ctypes.byref(k)) == 0
    want = oracle.bottom_up(o, f, w)
    assert k.value == want[0].size > 4
    assert fr.cpu().tolist() == [-7] * 4
    fr = torch.empty(k.value, dtype=torch.int32, device=dev)
    assert lib.cct_bottom_up(tree.handle, None, k.value, ctypes.c_void_p(fr.data_ptr()), None, None,
                             ctypes.byref(k)) == 0
    assert np.array_equal(fr.cpu().numpy().view(np.uint32), want[0])
    tree.free()


@pytest.mark.slow
@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["deep_recursion", "layered_16m"])
def test_view_full_size(name):
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.generate(name)
    print(f"{name}: N={o.size - 1:,} F={f.size:,}: building", flush=True)
    tree = cct.build(*to_dev(o, f, w))
    got = gpu_view(tree)
    tree.free()
    cct.release_cached_memory()
    print(f"{name}: view of {got[0].size:,} frames; oracle", flush=True)
    want = oracle.bottom_up(o, f, w)
    print(f"{name}: oracle done", flush=True)
    assert_view(got, want, name)
