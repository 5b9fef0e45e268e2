"""ORACLE — test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the bench's ``cpu_baseline`` leg
may import this package.  It is a plain, slow CPU calling context tree (a
``std::map`` trie, see ``oracle.cpp``) written from the paper's description of the
profiler's tree (Design, "Profiler", "Calling Context Tree"): call paths are
inserted with frames that name the same location collapsed, metrics are summed at
the node a path ends on (exclusive) and propagated to the root along the whole path
(inclusive).  It shares no code with the HIP path.

Readings fixed here (the paper is silent on them): frames are uint32 ids; the root
is the empty path with id 0, parent 0xFFFFFFFF, frame 0, depth 0; node ids are the
unsigned lexicographic rank of the root path (a proper prefix sorts first); sums are
uint64 modulo 2^64; a zero-length path adds to the root's exclusive sum.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None
NO_PARENT = 0xFFFFFFFF


def build(verbose: bool = False) -> str:
    """Compile liboracle.so in place (host C++, g++ -O2, single-threaded trie)."""
    src = os.path.join(_HERE, "oracle.cpp")
    tmp = _LIB_PATH + ".tmp"
    cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-pthread", src, "-o", tmp]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        lib.or_create.restype = vp
        lib.or_create.argtypes = [i32]
        lib.or_create_stats.restype = vp
        lib.or_create_stats.argtypes = [i32]
        lib.or_stats_export.argtypes = [vp, vp, vp, vp, vp, vp, vp]
        lib.or_destroy.argtypes = [vp]
        lib.or_destroy.restype = None
        lib.or_ingest.argtypes = [vp, i64, vp, vp, vp]
        lib.or_finalize.restype = i64
        lib.or_finalize.argtypes = [vp]
        lib.or_export.argtypes = [vp, vp, vp, vp, vp, vp]
        lib.or_brute.restype = i64
        lib.or_brute.argtypes = [i64, vp, vp, vp, i32, vp, vp, vp, vp, vp]
        lib.or_point_query.argtypes = [i64, vp, vp, vp, i32, i64, vp, vp, vp, vp, vp, ctypes.c_int]
        lib.or_check.argtypes = [i64, i32, vp, vp, vp, vp, vp, vp, vp]
        lib.or_bottom_up.restype = vp
        lib.or_bottom_up.argtypes = [i64, vp, vp, vp, i32]
        lib.or_bottom_up_size.restype = i64
        lib.or_bottom_up_size.argtypes = [vp]
        lib.or_bottom_up_fetch.argtypes = [vp, vp, vp, vp]
        lib.or_bottom_up_fetch.restype = None
        lib.or_bottom_up_free.argtypes = [vp]
        lib.or_bottom_up_free.restype = None
        _lib = lib
    return _lib


def _csr(offsets, frames, metrics, m=None):
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    frames = np.ascontiguousarray(frames, dtype=np.uint32)
    if frames.size == 0:
        frames = np.zeros(1, np.uint32)
    n = offsets.size - 1
    if metrics is None:
        metrics = np.zeros((n, m or 1), np.uint64)
    metrics = np.ascontiguousarray(metrics, dtype=np.uint64).reshape(n, -1) if n else \
        np.zeros((0, m or (metrics.shape[1] if metrics.ndim == 2 else 1)), np.uint64)
    return offsets, frames, metrics


class Tree(dict):
    """Canonical tree: keys parent, frame, depth (uint32[U]), excl, incl (uint64[U, M])."""

    @property
    def n_nodes(self):
        return int(self["parent"].size)


class Oracle:
    """Incremental std::map trie: ``ingest`` any number of CSR batches, then ``tree``."""

    def __init__(self, n_metrics, stats=False):
        self.m = int(n_metrics)
        self.stats = bool(stats)
        self._h = (_load().or_create_stats if self.stats else _load().or_create)(self.m)
        if not self._h:
            raise ValueError("bad metric count")

    def ingest(self, offsets, frames, metrics):
        o, f, w = _csr(offsets, frames, metrics, self.m)
        if w.shape[1] != self.m:
            raise ValueError("metric count mismatch")
        if _load().or_ingest(self._h, o.size - 1, _p(o), _p(f), _p(w)) != 0:
            raise ValueError("malformed offsets")

    def tree(self) -> Tree:
        lib = _load()
        U = lib.or_finalize(self._h)
        t = Tree(parent=np.empty(U, np.uint32), frame=np.empty(U, np.uint32), depth=np.empty(U, np.uint32),
                 excl=np.empty((U, self.m), np.uint64), incl=np.empty((U, self.m), np.uint64))
        lib.or_export(self._h, _p(t["parent"]), _p(t["frame"]), _p(t["depth"]), _p(t["excl"]), _p(t["incl"]))
        if self.stats:
            for k in ("count_excl", "count_incl"):
                t[k] = np.empty(U, np.uint64)
            for k in ("min_excl", "min_incl"):
                t[k] = np.empty((U, self.m), np.uint64)
            for k in ("sumsq_excl", "sumsq_incl"):
                t[k] = np.empty((U, self.m, 2), np.uint64)
            lib.or_stats_export(self._h, *(_p(t[k]) for k in ("count_excl", "count_incl", "min_excl", "min_incl",
                                                               "sumsq_excl", "sumsq_incl")))
        return t

    def close(self):
        if self._h:
            _load().or_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def build_tree(offsets, frames, metrics, stats=False) -> Tree:
    """One-shot oracle tree of a CSR trace (with per-node statistics if ``stats``)."""
    o, f, w = _csr(offsets, frames, metrics)
    orc = Oracle(w.shape[1], stats=stats)
    try:
        orc.ingest(o, f, w)
        return orc.tree()
    finally:
        orc.close()


def brute_tree(offsets, frames, metrics) -> Tree:
    """Brute-force prefix enumeration (tiny inputs only)."""
    o, f, w = _csr(offsets, frames, metrics)
    n, m = o.size - 1, w.shape[1]
    lib = _load()
    U = lib.or_brute(n, _p(o), _p(f), _p(w), m, None, None, None, None, None)
    if U < 0:
        raise ValueError("malformed offsets")
    t = Tree(parent=np.empty(U, np.uint32), frame=np.empty(U, np.uint32), depth=np.empty(U, np.uint32),
             excl=np.empty((U, m), np.uint64), incl=np.empty((U, m), np.uint64))
    lib.or_brute(n, _p(o), _p(f), _p(w), m, _p(t["parent"]), _p(t["frame"]), _p(t["depth"]),
                 _p(t["excl"]), _p(t["incl"]))
    return t


def point_query(offsets, frames, metrics, q_offsets, q_frames, threads=None):
    """(count[Q], excl[Q, M], incl[Q, M]) of query paths by a full scan of the events."""
    o, f, w = _csr(offsets, frames, metrics)
    qo = np.ascontiguousarray(q_offsets, dtype=np.int64)
    qf = np.ascontiguousarray(q_frames, dtype=np.uint32)
    if qf.size == 0:
        qf = np.zeros(1, np.uint32)
    nq, m = qo.size - 1, w.shape[1]
    cnt = np.empty(nq, np.int64)
    ex = np.empty((nq, m), np.uint64)
    inc = np.empty((nq, m), np.uint64)
    th = threads or max(1, min(16, len(os.sched_getaffinity(0))))
    if _load().or_point_query(o.size - 1, _p(o), _p(f), _p(w), m, nq, _p(qo), _p(qf), _p(cnt), _p(ex),
                              _p(inc), th) != 0:
        raise ValueError("malformed offsets")
    return cnt, ex, inc


CHECK_MESSAGES = {
    1: "root fields", 2: "parent id not smaller than node id", 3: "depth != parent depth + 1",
    4: "siblings not in strictly increasing frame order", 5: "ids are not a preorder",
    6: "inclusive != exclusive + sum of children's inclusive", 7: "root inclusive != total",
    8: "sum of exclusive != root inclusive",
}


def check(tree, total=None):
    """Run the invariant checker; returns (code, node) with code 0 when all hold."""
    parent = np.ascontiguousarray(tree["parent"], np.uint32)
    U = parent.size
    excl = np.ascontiguousarray(tree["excl"], np.uint64).reshape(U, -1)
    incl = np.ascontiguousarray(tree["incl"], np.uint64).reshape(U, -1)
    tot = None if total is None else np.ascontiguousarray(total, np.uint64)
    bad = np.zeros(1, np.int64)
    code = _load().or_check(U, excl.shape[1], _p(parent), _p(np.ascontiguousarray(tree["frame"], np.uint32)),
                            _p(np.ascontiguousarray(tree["depth"], np.uint32)), _p(excl), _p(incl),
                            _p(tot), _p(bad))
    return int(code), int(bad[0])


def total_metrics(metrics):
    """Column sums of uint64 metrics modulo 2^64."""
    w = np.asarray(metrics, np.uint64)
    if w.size == 0:
        return np.zeros(w.shape[1] if w.ndim == 2 else 1, np.uint64)
    return w.sum(axis=0, dtype=np.uint64)


def join_activity(reg_offsets, reg_frames, reg_corr_ids, corr_ids, metrics):
    """Correlation-ID join of one flush of activity records (Design, "Profiler", "GPU
    Metrics"): at each GPU API callback the profiler emits a unique correlation ID and
    associates it with the call path retrieved there; when the metric buffer is full,
    every flushed record is linked through its ID to that path and aggregated.

    Written from that definition: a dictionary from ID to registered path, then one
    event per record whose ID is registered, in record order, holding the registered
    path and the record's metrics.  Returns (offsets, frames, metrics, n_unmatched) of
    that CSR batch; ``Oracle.ingest`` of the batch is the merge.  An ID registered
    twice raises ValueError (the paper's IDs are unique)."""
    ro = np.asarray(reg_offsets, np.int64)
    rf = np.asarray(reg_frames, np.uint32)
    path_of = {}
    for i, c in enumerate(np.asarray(reg_corr_ids, np.uint64).tolist()):
        if c in path_of:
            raise ValueError(f"correlation ID {c} registered twice")
        path_of[c] = i
    w = np.asarray(metrics, np.uint64)
    if w.ndim < 2:
        w = w.reshape(-1, 1)
    rec, reg, unmatched = [], [], 0
    for r, c in enumerate(np.asarray(corr_ids, np.uint64).tolist()):
        i = path_of.get(c)
        if i is None:
            unmatched += 1
        else:
            rec.append(r)
            reg.append(i)
    reg = np.asarray(reg, np.int64)
    lens = ro[reg + 1] - ro[reg] if reg.size else np.zeros(0, np.int64)
    offsets = np.zeros(reg.size + 1, np.int64)
    np.cumsum(lens, out=offsets[1:])
    # frames of event k: the registered path reg[k], copied in event order
    starts = ro[reg] if reg.size else np.zeros(0, np.int64)
    pos = np.repeat(starts - offsets[:-1], lens) + np.arange(offsets[-1], dtype=np.int64)
    frames = rf[pos] if pos.size else np.zeros(0, np.uint32)
    return offsets, frames, w[np.asarray(rec, np.int64)].reshape(len(rec), w.shape[1]), unmatched


def join_activity_calls(reg_offsets, reg_frames, reg_corr_ids, corr_ids, metrics):
    """The same join with one event per API call rather than per record: every
    registered path that at least one record names, in registry order, carrying the sum
    (modulo 2^64) of its records' metrics.  Several records of one correlation ID report
    one call, so a tree keeping per-node statistics takes one sample per call.  For sums
    the two batches give the same tree.  Returns (offsets, frames, metrics, n_unmatched)."""
    o, f, w, unmatched = join_activity(reg_offsets, reg_frames, reg_corr_ids, corr_ids, metrics)
    ro = np.asarray(reg_offsets, np.int64)
    rf = np.asarray(reg_frames, np.uint32)
    index = {c: i for i, c in enumerate(np.asarray(reg_corr_ids, np.uint64).tolist())}
    m = w.shape[1]
    total = {}
    for c, row in zip(np.asarray(corr_ids, np.uint64).tolist(), np.asarray(metrics, np.uint64).reshape(-1, m).tolist()):
        i = index.get(c)
        if i is None:
            continue
        acc = total.setdefault(i, [0] * m)
        for j in range(m):
            acc[j] = (acc[j] + row[j]) % 2**64
    calls = sorted(total)
    offsets = np.zeros(len(calls) + 1, np.int64)
    frames, rows = [], []
    for k, i in enumerate(calls):
        frames.extend(rf[ro[i]:ro[i + 1]].tolist())
        offsets[k + 1] = len(frames)
        rows.append(total[i])
    return offsets, np.asarray(frames, np.uint32), np.asarray(rows, np.uint64).reshape(len(calls), m), unmatched


def bottom_up(offsets, frames, metrics):
    """Bottom-up view from the events (``or_bottom_up`` in oracle.cpp): for every frame on
    some path, ascending, (frames[K], excl[K, M], incl[K, M]) where excl sums the events
    whose path ends with the frame and incl the events whose path contains it, each event
    once however often the frame recurs (Implementation, "GUI": the bottom-up view
    aggregates the metrics of the same node across different call paths)."""
    o, f, w = _csr(offsets, frames, metrics)
    n, m = o.size - 1, w.shape[1]
    lib = _load()
    h = lib.or_bottom_up(n, _p(o), _p(f), _p(w), m)
    if not h:
        raise ValueError("malformed offsets")
    try:
        K = lib.or_bottom_up_size(h)
        fr = np.empty(max(K, 1), np.uint32)
        ex = np.empty((max(K, 1), m), np.uint64)
        inc = np.empty((max(K, 1), m), np.uint64)
        lib.or_bottom_up_fetch(h, _p(fr), _p(ex), _p(inc))
    finally:
        lib.or_bottom_up_free(h)
    return fr[:K], ex[:K], inc[:K]


def filter_nodes(tree, num_metric, op, thr_num, thr_den, num_excl=False, den="one", den_metric=0, den_excl=False,
                 leaves_only=False):
    """Node ids whose metric ratio crosses a threshold, ascending (the example analyses
    flag nodes whose ratio of metrics is above or below a threshold: Implementation,
    "Performance Analyzer", "Example Analyses").  Reading fixed here: a / b above p / q
    means a * q > p * b (below: <), in exact integers, so no division; a is the node's
    incl (or excl) sum of num_metric; b is 1, the node's sum of den_metric, or the root's
    incl sum of den_metric; leaves_only keeps nodes that are nobody's parent."""
    parent = tree["parent"]
    U = parent.size
    a = [int(x) for x in tree["excl" if num_excl else "incl"][:, num_metric]]
    if den == "one":
        b = [1] * U
    elif den == "metric":
        b = [int(x) for x in tree["excl" if den_excl else "incl"][:, den_metric]]
    else:
        b = [int(tree["incl"][0, den_metric])] * U
    parents = set(int(p) for p in parent[1:])
    p, q = int(thr_num), int(thr_den)
    out = []
    for v in range(U):
        lhs, rhs = a[v] * q, p * b[v]
        if (lhs > rhs if op > 0 else lhs < rhs) and not (leaves_only and v in parents):
            out.append(v)
    return np.asarray(out, np.int64)


def derived_stats(tree, nodes=None):
    """Mean and standard deviation of every metric at the given nodes (all by default),
    exclusive and inclusive, from a statistics tree (``build_tree(..., stats=True)``).

    The paper keeps sum, minimum, average and standard deviation per node metric
    (Design, "Profiler", "Calling Context Tree").  Readings fixed here: the average is
    sum / count over the node's samples (the events ending at the node, or passing
    through it); the standard deviation is the population one, sqrt(n * S2 - S1^2) / n
    with S1 the node's sum (modulo 2^64, as the tree keeps it) and S2 its sum of squares
    (modulo 2^128); both are NaN where the count is 0, and the deviation is NaN where
    n * S2 - S1^2 is negative (possible only when a sum wrapped).  Each value is the
    exact quantity rounded once to float64 (Fraction for the mean, 60-digit Decimal
    square root for the deviation)."""
    from decimal import Context
    from fractions import Fraction
    ctx = Context(prec=60)
    U, m = tree["parent"].size, tree["excl"].shape[1]
    idx = np.arange(U) if nodes is None else np.asarray(nodes, np.int64)
    out = {}
    for side in ("excl", "incl"):
        mean = np.full((idx.size, m), np.nan)
        std = np.full((idx.size, m), np.nan)
        for r, v in enumerate(idx):
            n = int(tree["count_" + side][v])
            if n == 0:
                continue
            for j in range(m):
                s1 = int(tree[side][v, j])
                lo, hi = (int(x) for x in tree["sumsq_" + side][v, j])
                s2 = lo | (hi << 64)
                mean[r, j] = float(Fraction(s1, n))
                d = n * s2 - s1 * s1
                if d >= 0:
                    std[r, j] = float(ctx.divide(ctx.sqrt(ctx.create_decimal(d)), ctx.create_decimal(n)))
        out["mean_" + side], out["std_" + side] = mean, std
    return out
