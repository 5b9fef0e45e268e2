"""cct_filter_noalloc (the ratio filter that allocates nothing: its scratch is a static
device array) against cct_filter and the oracle, through the C ABI: the same node ids
and counts on two calls in a row, the second on a smaller tree, so that the static
array's leftovers from the first call cannot leak into the second."""
import ctypes

import numpy as np
import pytest

import oracle
import tracegen
from gpu_util import to_dev, torch_or_skip

pytestmark = pytest.mark.gpu


def run_filter(lib, fn, tree, spec, capacity):
    import torch
    out = torch.full((max(capacity, 1),), -7, dtype=torch.int64, device="cuda")
    k = ctypes.c_int64(-1)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    st = getattr(lib, fn)(tree.handle, ctypes.byref(spec), stream, capacity,
                          ctypes.c_void_p(out.data_ptr()), ctypes.byref(k))
    assert st == 0, (fn, st, lib.cct_last_error())
    return out[:min(k.value, capacity)].cpu().numpy(), k.value


SPECS = [  # (num_metric, num_excl, den_kind, den_metric, den_excl, op, thr_num, thr_den, leaves_only)
    (0, 0, 2, 0, 0, +1, 1, 200, 1),   # hotspot leaves
    (0, 0, 1, 1, 0, -1, 5, 1, 0),     # small kernels
    (2, 0, 1, 0, 0, +1, 1, 4, 0),     # CPU latency
    (1, 1, 0, 0, 0, +1, 0, 1, 0),     # any nonzero exclusive sum
]


def test_noalloc_filter_matches_allocating_filter_twice():
    torch_or_skip()
    import paper_2411_02797_amd as cct
    lib = cct.load_library()
    for seed, n in ((11, 20000), (12, 3000)):  # second call on a smaller tree
        o, f, w = tracegen.random_paths(n, 40, 20, 3, seed=seed)
        tree = cct.build(*to_dev(o, f, w))
        want_tree = oracle.build_tree(o, f, w)
        u = tree.n_nodes
        assert u > 2048 * 2 or n < 10000  # the larger tree spans several filter tiles
        for spec_t in SPECS:
            spec = cct._FilterSpec(*spec_t)
            want_ids = oracle.filter_nodes(want_tree, spec_t[0], spec_t[5], spec_t[6], spec_t[7],
                                           num_excl=bool(spec_t[1]), den=("one", "metric", "root")[spec_t[2]],
                                           den_metric=spec_t[3], den_excl=bool(spec_t[4]),
                                           leaves_only=bool(spec_t[8]))
            for cap in (u, max(len(want_ids) // 2, 1), 0):
                got, k = run_filter(lib, "cct_filter_noalloc", tree, spec, cap)
                ref, k_ref = run_filter(lib, "cct_filter", tree, spec, cap)
                assert k == k_ref == len(want_ids), (seed, spec_t, cap, k, k_ref, len(want_ids))
                assert np.array_equal(got, ref), (seed, spec_t, cap)
                assert np.array_equal(got, want_ids[:cap]), (seed, spec_t, cap)
        tree.free()


def test_noalloc_filter_rejects_bad_arguments():
    torch_or_skip()
    import paper_2411_02797_amd as cct
    lib = cct.load_library()
    o, f, w = tracegen.random_paths(500, 10, 8, 1, seed=5)
    tree = cct.build(*to_dev(o, f, w))
    k = ctypes.c_int64(-1)
    bad = cct._FilterSpec(3, 0, 0, 0, 0, +1, 1, 1, 0)  # metric 3 of a one-metric tree
    assert lib.cct_filter_noalloc(tree.handle, ctypes.byref(bad), None, 0, None,
                                  ctypes.byref(k)) == -1
    assert k.value == -1  # untouched on error
    tree.free()
