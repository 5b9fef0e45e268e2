"""Helpers for the GPU tests: move CSR traces to the device, run the library, compare
with the oracle."""
import numpy as np
import pytest

FIELDS = ("parent", "frame", "depth", "excl", "incl")


def torch_or_skip():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def to_dev(o, f, w):
    torch = torch_or_skip()
    dev = torch.device("cuda", 0)
    to = torch.from_numpy(np.ascontiguousarray(o, np.int64)).to(dev)
    fa = np.ascontiguousarray(f, np.uint32)
    tf = torch.from_numpy(fa.view(np.int32)).to(dev) if fa.size else torch.zeros(0, dtype=torch.int32, device=dev)
    wa = np.ascontiguousarray(w, np.uint64)
    tw = torch.from_numpy(wa.view(np.int64).reshape(wa.shape)).to(dev)
    return to, tf, tw


def gpu_tree(o, f, w):
    import paper_2411_02797_amd as cct
    tree = cct.build(*to_dev(o, f, w))
    try:
        return tree.to_numpy()
    finally:
        tree.free()


def assert_same(got, want, ctx=""):
    for k in FIELDS:
        g = np.asarray(got[k])
        x = np.asarray(want[k])
        g = g.reshape(x.shape) if g.size == x.size else g
        assert g.shape == x.shape, f"{ctx}: {k} shape {g.shape} vs {x.shape}"
        if not np.array_equal(g, x):
            bad = np.flatnonzero((g != x).ravel())
            raise AssertionError(f"{ctx}: {k} differs at {bad[:8]} (of {bad.size}); got {g.ravel()[bad[:4]]} "
                                 f"want {x.ravel()[bad[:4]]}")


def node_paths(tree, nodes):
    """Root paths of the given node ids, reconstructed from parent/frame arrays."""
    parent, frame = tree["parent"], tree["frame"]
    out = []
    for v in nodes:
        p = []
        v = int(v)
        while v != 0:
            p.append(int(frame[v]))
            v = int(parent[v])
        out.append(p[::-1])
    return out


def csr(paths):
    o = np.zeros(len(paths) + 1, np.int64)
    o[1:] = np.cumsum([len(p) for p in paths])
    f = np.array([x for p in paths for x in p], np.uint32)
    return o, f
