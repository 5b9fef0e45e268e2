import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU; runs through the C ABI")
    config.addinivalue_line("markers", "slow: full-size workloads")


def load_golden(name):
    """Parse a tests/golden/*.txt fixture -> (offsets, frames, metrics, expected tree)."""
    import numpy as np
    path = os.path.join(ROOT, "tests", "golden", name)
    m = None
    paths, ws, nodes = [], [], []
    with open(path) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            tag, rest = line.split(None, 1)
            if tag == "M":
                m = int(rest)
            elif tag == "E":
                p, w = [s.strip() for s in rest.split("|")]
                paths.append([] if p == "-" else [int(x) for x in p.split(",")])
                ws.append([int(x) for x in w.split(",")])
            elif tag == "N":
                head, ex, inc = [s.strip() for s in rest.split("|")]
                par, fr, dp = head.split()
                nodes.append((0xFFFFFFFF if par == "-" else int(par), int(fr), int(dp),
                              [int(x) for x in ex.split(",")], [int(x) for x in inc.split(",")]))
    offsets = np.zeros(len(paths) + 1, np.int64)
    offsets[1:] = np.cumsum([len(p) for p in paths])
    frames = np.array([x for p in paths for x in p], dtype=np.uint32)
    metrics = np.array(ws, dtype=np.uint64).reshape(len(paths), m)
    tree = {
        "parent": np.array([n[0] for n in nodes], np.uint32),
        "frame": np.array([n[1] for n in nodes], np.uint32),
        "depth": np.array([n[2] for n in nodes], np.uint32),
        "excl": np.array([n[3] for n in nodes], np.uint64).reshape(len(nodes), m),
        "incl": np.array([n[4] for n in nodes], np.uint64).reshape(len(nodes), m),
    }
    return offsets, frames, metrics, tree
