"""Seeded synthetic call-path traces in CSR form.

Shared by the CPU oracle tests and the GPU path: this module holds the workload
recipes only, none of the calling-context-tree arithmetic.  Every trace is
``(offsets int64[N+1], frames uint32[F], metrics uint64[N, M])`` with each path
root-first (outermost caller first, GPU-kernel leaf last), the shape the paper's
call-path integration produces (Design, "Call Path Integration").
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libtracegen.so")
_lib = None

# name -> (kind, default events, seed, seed2, p0, p1, p2)
WORKLOADS = {
    # 10,000 events on a random recursive call-site tree (2,000 labels, depth <= 16)
    "tiny": (0, 10_000, 1001, 0, 0, 0, 0),
    # 1M events, layered Python/framework/C++/kernel ids (50,000), depth 8..64, 3 metrics
    "layered_1m": (1, 1 << 20, 1002, 0, 0, 0, 0),
    # 16M events, 200,000 ids, depth 16..128, 90% under 8 training-loop roots, 2 metrics
    "layered_16m": (2, 1 << 24, 1003, 0, 0, 0, 0),
    # 8M-event base of the incremental merge, 4 metrics (last one full-range)
    "merge_base": (3, 1 << 23, 1004, 0, 0, 0, 0),
    # 2M-event merge chunk (p0 = chunk index 0..31), events from seed 2004 + chunk
    "merge_chunk": (4, 1 << 21, 1004, 2004, 0, 0, 0),
    # 4M events, depth 256..512 recursion of a 12-frame cycle + 1% single frames
    "deep_recursion": (5, 1 << 22, 1005, 0, 0, 0, 0),
}


def build(verbose: bool = False) -> str:
    """Compile libtracegen.so in place (host C++, g++)."""
    src = os.path.join(_HERE, "tracegen.cpp")
    tmp = _LIB_PATH + ".tmp"
    cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-pthread", src, "-o", tmp]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        lib.tg_create.restype = ctypes.c_void_p
        lib.tg_create.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint64,
                                  ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int]
        lib.tg_n_frames.restype = ctypes.c_int64
        lib.tg_n_frames.argtypes = [ctypes.c_void_p]
        lib.tg_n_metrics.restype = ctypes.c_int32
        lib.tg_n_metrics.argtypes = [ctypes.c_void_p]
        lib.tg_fill.restype = ctypes.c_int
        lib.tg_fill.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_int]
        lib.tg_destroy.restype = None
        lib.tg_destroy.argtypes = [ctypes.c_void_p]
        _lib = lib
    return _lib


def _threads(threads):
    if threads:
        return int(threads)
    return max(1, min(16, len(os.sched_getaffinity(0))))


def generate_kind(kind, n_events, seed, seed2=0, p0=0, p1=0, p2=0, threads=None, out=None):
    """Generate one trace.  ``out`` may hold preallocated (offsets, frames, metrics)
    arrays (e.g. pinned host memory viewed as numpy) of the right sizes."""
    lib = _load()
    th = _threads(threads)
    h = lib.tg_create(kind, n_events, seed, seed2, p0, p1, p2, th)
    if not h:
        raise ValueError("tracegen: bad arguments")
    try:
        nf = lib.tg_n_frames(h)
        m = lib.tg_n_metrics(h)
        if out is None:
            offsets = np.empty(n_events + 1, dtype=np.int64)
            frames = np.empty(max(nf, 1), dtype=np.uint32)[:nf]
            metrics = np.empty((n_events, m), dtype=np.uint64)
        else:
            offsets, frames, metrics = out
        fr_ptr = frames.ctypes.data if nf > 0 else np.empty(1, np.uint32).ctypes.data
        rc = lib.tg_fill(h, offsets.ctypes.data, fr_ptr, metrics.ctypes.data if n_events else None, th)
        if rc != 0:
            raise RuntimeError("tracegen: fill failed")
        return offsets, frames, metrics
    finally:
        lib.tg_destroy(h)


def sizes(name, n_events=None, chunk=0):
    """(n_events, n_frames, n_metrics) of a named workload without materialising it."""
    kind, n0, seed, seed2, p0, p1, p2 = WORKLOADS[name]
    n = n0 if n_events is None else int(n_events)
    lib = _load()
    h = lib.tg_create(kind, n, seed, seed2, chunk if kind == 4 else p0, p1, p2, _threads(None))
    if not h:
        raise ValueError("tracegen: bad arguments")
    try:
        return n, lib.tg_n_frames(h), lib.tg_n_metrics(h)
    finally:
        lib.tg_destroy(h)


def generate(name, n_events=None, chunk=0, threads=None, out=None):
    """Generate a named workload (see ``WORKLOADS``); ``n_events`` scales it down."""
    kind, n0, seed, seed2, p0, p1, p2 = WORKLOADS[name]
    n = n0 if n_events is None else int(n_events)
    if kind == 4:
        p0 = int(chunk)
    return generate_kind(kind, n, seed, seed2, p0, p1, p2, threads=threads, out=out)


def random_small(n_events, alphabet, max_len, n_metrics, seed, threads=1):
    """Tiny random traces over <= 16 special ids (0, 0x7FFFFFFF, 0x80000000,
    0xFFFFFFFF, ...), lengths 0..max_len, full-range uint64 metrics."""
    return generate_kind(6, n_events, seed, 0, alphabet, max_len, n_metrics, threads=threads)


def random_paths(n_events, n_ids, max_len, n_metrics, seed, threads=None):
    """Random paths over an ``n_ids`` pool, lengths 1..max_len, metrics < 2^20."""
    return generate_kind(7, n_events, seed, 0, n_ids, max_len, n_metrics, threads=threads)
