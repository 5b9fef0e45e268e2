"""Seeded input generators: reproducible, thread-count independent, right shapes."""
import numpy as np
import pytest

import tracegen


@pytest.mark.parametrize("name,n", [("tiny", None), ("layered_1m", 50_000), ("layered_16m", 20_000),
                                    ("merge_base", 20_000), ("merge_chunk", 20_000),
                                    ("deep_recursion", 5_000)])
def test_deterministic_and_thread_independent(name, n):
    a = tracegen.generate(name, n_events=n, threads=1)
    b = tracegen.generate(name, n_events=n, threads=7)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    o, f, w = a
    assert o[0] == 0 and np.all(np.diff(o) >= 0) and o[-1] == f.size


def test_shapes_of_the_workloads():
    o, f, w = tracegen.generate("tiny")
    L = np.diff(o)
    assert o.size == 10_001 and w.shape == (10_000, 1) and L.min() >= 1 and L.max() <= 16
    assert np.unique(f).size <= 2000 and w.min() >= 1000 and w.max() <= 1_000_000
    o, f, w = tracegen.generate("layered_16m", n_events=30_000)
    L = np.diff(o)
    assert w.shape == (30_000, 2) and L.min() >= 16 and L.max() <= 128
    o, f, w = tracegen.generate("deep_recursion", n_events=20_000)
    L = np.diff(o)
    assert L.max() <= 512 and np.mean(L == 1) > 0.005 and np.mean(L == 1) < 0.02
    assert np.all((L == 1) | (L >= 256))
    o, f, w = tracegen.generate("merge_chunk", n_events=10_000, chunk=3)
    assert w.shape == (10_000, 4) and w[:, 1].max() == 1 and w[:, 3].max() > 2**62


def test_chunks_differ_and_share_program():
    a = tracegen.generate("merge_chunk", n_events=5_000, chunk=0)
    b = tracegen.generate("merge_chunk", n_events=5_000, chunk=1)
    assert not np.array_equal(a[1][:1000], b[1][:1000])


def test_random_small_special_ids():
    o, f, w = tracegen.random_small(2000, 16, 8, 2, seed=1)
    assert set(np.unique(f).tolist()) >= {0, 0xFFFFFFFF, 0x80000000, 0x7FFFFFFF}
    assert np.diff(o).min() == 0
