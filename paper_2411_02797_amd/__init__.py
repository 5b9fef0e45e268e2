"""Calling context tree construction on one AMD MI355X (gfx950).

Thin ctypes binding over ``libcct.so`` (see ``include/cct.h``): argument marshalling
only, every step of the tree construction runs in the library's HIP kernels.  PyTorch
provides device memory and the current stream.  If ``libcct.so`` is missing or fails
to load, every call raises; there is no CPU fallback.

    tree = build(offsets, frames, metrics)   # int64[N+1], int32/uint32[F], int64/uint64[N, M]
    tree.merge(offsets2, frames2, metrics2)  # aggregate one more batch
    unmatched = tree.merge_activity(reg_offsets, reg_frames, reg_corr_ids, corr_ids, metrics3)
    ids, excl, incl = tree.query(q_offsets, q_frames)
    arrays = tree.to_tensors()               # parent, frame, depth, excl, incl on the GPU
    view = tree.bottom_up()                  # frames, excl, incl per distinct frame
    ids = tree.filter(0, +1, 1, 100, den="root", leaves_only=True)  # hotspots above 1% of the root
"""
from __future__ import annotations

import ctypes
import os

__all__ = ["build", "Tree", "CctError", "library_path", "load_library", "last_timings", "release_cached_memory",
           "EXPORTED_SYMBOLS", "NO_PARENT"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libcct.so")
_lib = None

NO_PARENT = 0xFFFFFFFF
MAX_METRICS = 8
EXPORTED_SYMBOLS = ("cct_build", "cct_build_stats", "cct_stats", "cct_merge", "cct_merge_activity", "cct_bottom_up", "cct_filter", "cct_filter_noalloc", "cct_query",
                    "cct_info", "cct_export", "cct_free", "cct_release_cached_memory", "cct_last_error",
                    "cct_last_timings")
_STATUS = {0: "CCT_OK", -1: "CCT_EINVAL", -2: "CCT_ENOMEM", -3: "CCT_EDEVICE", -4: "CCT_EMISMATCH",
           -5: "CCT_EOVERFLOW"}


class CctError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        self.name = _STATUS.get(status, str(status))
        super().__init__(f"{self.name}: {message}")


class _Paths(ctypes.Structure):
    _fields_ = [("n_events", ctypes.c_int64), ("n_frames", ctypes.c_int64), ("n_metrics", ctypes.c_int32),
                ("offsets", ctypes.c_void_p), ("frames", ctypes.c_void_p), ("metrics", ctypes.c_void_p)]


class _Activity(ctypes.Structure):
    _fields_ = [("n_records", ctypes.c_int64), ("n_metrics", ctypes.c_int32), ("corr_ids", ctypes.c_void_p),
                ("metrics", ctypes.c_void_p)]


class _FilterSpec(ctypes.Structure):
    _fields_ = [("num_metric", ctypes.c_int32), ("num_excl", ctypes.c_int32), ("den_kind", ctypes.c_int32),
                ("den_metric", ctypes.c_int32), ("den_excl", ctypes.c_int32), ("op", ctypes.c_int32),
                ("thr_num", ctypes.c_uint64), ("thr_den", ctypes.c_uint64), ("leaves_only", ctypes.c_int32)]


_DEN_KINDS = {"one": 0, "metric": 1, "root": 2}

_STAT_FIELDS = ("count_excl", "count_incl", "min_excl", "min_incl", "sumsq_excl", "sumsq_incl", "mean_excl",
                "mean_incl", "std_excl", "std_incl")


class _NodeStats(ctypes.Structure):
    _fields_ = [(k, ctypes.c_void_p) for k in _STAT_FIELDS]


def library_path():
    return _LIB_PATH


def load_library():
    """Load libcct.so (built by ``__graft_entry__.build()``); raises if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: run __graft_entry__.build() (hipcc, gfx950) first")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    P = ctypes.POINTER
    lib.cct_build.argtypes = [P(_Paths), vp, P(vp)]
    lib.cct_build_stats.argtypes = [P(_Paths), vp, P(vp)]
    lib.cct_stats.argtypes = [vp, vp, P(_NodeStats)]
    lib.cct_merge.argtypes = [vp, P(_Paths), vp]
    lib.cct_merge_activity.argtypes = [vp, P(_Paths), vp, P(_Activity), vp, P(i64)]
    lib.cct_bottom_up.argtypes = [vp, vp, i64, vp, vp, vp, P(i64)]
    lib.cct_filter.argtypes = [vp, P(_FilterSpec), vp, i64, vp, P(i64)]
    lib.cct_filter_noalloc.argtypes = [vp, P(_FilterSpec), vp, i64, vp, P(i64)]
    lib.cct_query.argtypes = [vp, P(_Paths), vp, vp, vp, vp]
    lib.cct_info.argtypes = [vp, P(i64), P(i32), P(i64)]
    lib.cct_export.argtypes = [vp, vp, vp, vp, vp, vp, vp]
    lib.cct_free.argtypes = [vp]
    lib.cct_free.restype = None
    lib.cct_release_cached_memory.argtypes = []
    lib.cct_release_cached_memory.restype = None
    lib.cct_last_error.restype = ctypes.c_char_p
    lib.cct_last_timings.argtypes = [P(ctypes.c_double), ctypes.c_int]
    for name in ("cct_build", "cct_build_stats", "cct_stats", "cct_merge", "cct_merge_activity", "cct_bottom_up", "cct_filter", "cct_filter_noalloc", "cct_query",
                 "cct_info", "cct_export"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status):
    if status != 0:
        raise CctError(status, load_library().cct_last_error().decode())


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _paths(offsets, frames, metrics, need_metrics=True):
    import torch
    if not (offsets.is_cuda and frames.is_cuda):
        raise ValueError("offsets and frames must be device tensors")
    if offsets.dtype != torch.int64 or offsets.dim() != 1 or not offsets.is_contiguous():
        raise ValueError("offsets must be a contiguous int64[N+1] tensor")
    if frames.dtype not in (torch.int32, torch.uint32) or frames.dim() != 1 or not frames.is_contiguous():
        raise ValueError("frames must be a contiguous int32/uint32[F] tensor")
    n = offsets.numel() - 1
    if n < 0:
        raise ValueError("offsets must hold N+1 >= 1 elements")
    m = 1
    mp = None
    if metrics is not None:
        if not metrics.is_cuda or metrics.dtype not in (torch.int64, torch.uint64) or not metrics.is_contiguous():
            raise ValueError("metrics must be a contiguous int64/uint64 [N, M] device tensor")
        if metrics.dim() == 1:
            metrics = metrics.view(-1, 1)
        if metrics.shape[0] != n:
            raise ValueError("metrics must have N rows")
        m = metrics.shape[1]
        mp = metrics.data_ptr() if metrics.numel() else None
    elif need_metrics:
        raise ValueError("metrics required")
    p = _Paths(n, frames.numel(), m, offsets.data_ptr(), frames.data_ptr() if frames.numel() else None, mp)
    return p, m


class Tree:
    """A calling context tree owned by libcct (device memory, canonical node ids)."""

    def __init__(self, handle):
        self._h = ctypes.c_void_p(handle)

    @property
    def handle(self):
        return self._h

    def _info(self):
        u, m, d = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int64()
        _check(load_library().cct_info(self._h, ctypes.byref(u), ctypes.byref(m), ctypes.byref(d)))
        return u.value, m.value, d.value

    @property
    def n_nodes(self):
        return self._info()[0]

    @property
    def n_metrics(self):
        return self._info()[1]

    @property
    def n_paths(self):
        return self._info()[2]

    def merge(self, offsets, frames, metrics):
        p, _ = _paths(offsets, frames, metrics)
        _check(load_library().cct_merge(self._h, ctypes.byref(p), _stream()))
        return self

    def merge_activity(self, reg_offsets, reg_frames, reg_corr_ids, corr_ids, metrics):
        """Merge one activity flush (cct_merge_activity): record r (correlation ID
        corr_ids[r], metrics[r]) is linked to the registered path whose ID equals
        corr_ids[r] (reg_offsets/reg_frames CSR, IDs reg_corr_ids).  IDs are int64 or
        uint64 device tensors.  Returns the number of records with an unregistered ID."""
        import torch
        p, _ = _paths(reg_offsets, reg_frames, None, need_metrics=False)
        for name, t in (("reg_corr_ids", reg_corr_ids), ("corr_ids", corr_ids)):
            if not t.is_cuda or t.dtype not in (torch.int64, torch.uint64) or t.dim() != 1 or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous int64/uint64 device vector")
        if reg_corr_ids.numel() != p.n_events:
            raise ValueError("reg_corr_ids must have one ID per registered path")
        if not metrics.is_cuda or metrics.dtype not in (torch.int64, torch.uint64) or not metrics.is_contiguous():
            raise ValueError("metrics must be a contiguous int64/uint64 [R, M] device tensor")
        if metrics.dim() == 1:
            metrics = metrics.view(-1, 1)
        r = corr_ids.numel()
        if metrics.shape[0] != r:
            raise ValueError("metrics must have one row per record")
        act = _Activity(r, metrics.shape[1], corr_ids.data_ptr() if r else None, metrics.data_ptr() if r else None)
        un = ctypes.c_int64(0)
        _check(load_library().cct_merge_activity(self._h, ctypes.byref(p),
                                                 reg_corr_ids.data_ptr() if p.n_events else None,
                                                 ctypes.byref(act), _stream(), ctypes.byref(un)))
        return un.value

    def query(self, offsets, frames, want_metrics=True):
        import torch
        p, _ = _paths(offsets, frames, None, need_metrics=False)
        u, m, d = self._info()
        q = offsets.numel() - 1
        dev = offsets.device
        ids = torch.empty(max(q, 1), dtype=torch.int64, device=dev)[:q]
        ex = torch.empty((q, m), dtype=torch.int64, device=dev) if want_metrics else None
        inc = torch.empty((q, m), dtype=torch.int64, device=dev) if want_metrics else None
        _check(load_library().cct_query(self._h, ctypes.byref(p), _stream(), ids.data_ptr() if q else None,
                                        ex.data_ptr() if want_metrics and q else None,
                                        inc.data_ptr() if want_metrics and q else None))
        return ids, ex, inc

    def bottom_up(self, device=None):
        """Bottom-up view (cct_bottom_up): {"frames": int32[K] (bit patterns of uint32,
        ascending as unsigned), "excl", "incl": int64[K, M] (bit patterns of uint64)}."""
        import torch
        lib = load_library()
        k = ctypes.c_int64(0)
        _check(lib.cct_bottom_up(self._h, _stream(), 0, None, None, None, ctypes.byref(k)))
        u, m, _ = self._info()
        dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        out = {"frames": torch.empty(k.value, dtype=torch.int32, device=dev),
               "excl": torch.empty((k.value, m), dtype=torch.int64, device=dev),
               "incl": torch.empty((k.value, m), dtype=torch.int64, device=dev)}
        if k.value:
            _check(lib.cct_bottom_up(self._h, _stream(), k.value, out["frames"].data_ptr(), out["excl"].data_ptr(),
                                     out["incl"].data_ptr(), ctypes.byref(k)))
        return out

    def filter(self, num_metric, op, thr_num, thr_den, num_excl=False, den="one", den_metric=0, den_excl=False,
               leaves_only=False, noalloc=False):
        """Node ids matching a ratio test (cct_filter), ascending, as an int64 device
        tensor: a / b above (op=+1) or below (op=-1) thr_num / thr_den, with a the node's
        incl (or excl) sum of num_metric and b = 1 (den="one"), the node's sum of den_metric
        (den="metric") or the root's incl sum of den_metric (den="root").  noalloc=True
        calls cct_filter_noalloc (the library allocates nothing; the output tensor is still
        allocated here)."""
        import torch
        spec = _FilterSpec(num_metric, int(bool(num_excl)), _DEN_KINDS[den], den_metric, int(bool(den_excl)), op,
                           thr_num, thr_den, int(bool(leaves_only)))
        u = self.n_nodes
        out = torch.empty(max(u, 1), dtype=torch.int64, device=torch.device("cuda", torch.cuda.current_device()))
        k = ctypes.c_int64(0)
        fn = load_library().cct_filter_noalloc if noalloc else load_library().cct_filter
        _check(fn(self._h, ctypes.byref(spec), _stream(), u, out.data_ptr(), ctypes.byref(k)))
        return out[:k.value]

    def hotspots(self, time_metric, thr_num, thr_den):
        """Leaves whose inclusive time is above thr_num / thr_den of the root's (the paper's
        hotspot identification)."""
        return self.filter(time_metric, +1, thr_num, thr_den, den="root", den_metric=time_metric, leaves_only=True)

    def small_kernels(self, time_metric, count_metric, thr_num, thr_den):
        """Nodes whose inclusive time per launch is below thr_num / thr_den (the paper's
        kernel fusion analysis)."""
        return self.filter(time_metric, -1, thr_num, thr_den, den="metric", den_metric=count_metric)

    def cpu_latency(self, cpu_metric, gpu_metric, thr_num, thr_den):
        """Nodes whose inclusive CPU time is above thr_num / thr_den of their GPU time (the
        paper's CPU latency analysis)."""
        return self.filter(cpu_metric, +1, thr_num, thr_den, den="metric", den_metric=gpu_metric)

    def stats(self, device=None, fields=_STAT_FIELDS):
        """Per-node statistics (cct_stats) as tensors: count_* int64[U], min_* int64[U, M],
        sumsq_* int64[U, M, 2] (bit patterns of uint64; low word first), mean_* and std_*
        float64[U, M].  Only the named fields are computed into tensors."""
        import torch
        u, m, _ = self._info()
        dev = torch.device("cuda", torch.cuda.current_device())
        shapes = {"count": (u,), "min": (u, m), "sumsq": (u, m, 2), "mean": (u, m), "std": (u, m)}
        out = {}
        for k in fields:
            kind = k.split("_")[0]
            out[k] = torch.empty(shapes[kind], dtype=torch.float64 if kind in ("mean", "std") else torch.int64,
                                 device=dev)
        spec = _NodeStats(**{k: (out[k].data_ptr() if k in out else None) for k in _STAT_FIELDS})
        _check(load_library().cct_stats(self._h, _stream(), ctypes.byref(spec)))
        if device is not None:
            out = {k: v.to(device) for k, v in out.items()}
        return out

    def to_tensors(self, device=None):
        """Canonical arrays as tensors: parent/frame/depth int32[U] (bit patterns of
        uint32), excl/incl int64[U, M] (bit patterns of uint64)."""
        import torch
        u, m, _ = self._info()
        dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        out = {k: torch.empty(u, dtype=torch.int32, device=dev) for k in ("parent", "frame", "depth")}
        out["excl"] = torch.empty((u, m), dtype=torch.int64, device=dev)
        out["incl"] = torch.empty((u, m), dtype=torch.int64, device=dev)
        _check(load_library().cct_export(self._h, _stream(), *(out[k].data_ptr() for k in
                                                                ("parent", "frame", "depth", "excl", "incl"))))
        return out

    def to_numpy(self):
        """Canonical arrays as numpy (uint32 / uint64)."""
        import numpy as np
        t = self.to_tensors(device="cpu")
        return {k: (v.numpy().view(np.uint32) if v.dtype.itemsize == 4 else v.numpy().view(np.uint64))
                for k, v in t.items()}

    def free(self):
        if self._h is not None and self._h.value:
            load_library().cct_free(self._h)
        self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def build(offsets, frames, metrics, stats=False):
    """Build a calling context tree from one CSR batch of device tensors; with
    ``stats=True`` the tree also keeps per-node counts, minima and sums of squares
    (cct_build_stats), read with ``Tree.stats``."""
    p, _ = _paths(offsets, frames, metrics)
    h = ctypes.c_void_p()
    lib = load_library()
    _check((lib.cct_build_stats if stats else lib.cct_build)(ctypes.byref(p), _stream(), ctypes.byref(h)))
    return Tree(h.value)


def last_timings():
    """Per-phase HIP-event times (ms) of this thread's last calls: ingest, publish, sort,
    canonical emission and total of the last build/merge, the correlation-ID join of a
    merge_activity call (0 otherwise), the most recent computation of a bottom-up view
    (bottom_up), the last filter, the statistics kept by the last build/merge (0 without),
    the last ``Tree.stats``, the last query's lookups, and the prefix index it built (0 if
    the tree's index was kept)."""
    buf = (ctypes.c_double * 12)()
    n = load_library().cct_last_timings(buf, 12)
    return list(buf)[:n]


def release_cached_memory():
    """Return the library's cached device buffers to the HIP runtime (cct_release_cached_memory)."""
    load_library().cct_release_cached_memory()
