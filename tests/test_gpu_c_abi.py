"""The C ABI from a plain C program (tests/c_abi/cct_c_example.c, compiled here with gcc
against libcct.so and the HIP runtime, no Python or torch in the process): its build of the
hand-worked tree W1, a merge, and two lookups are compared with the golden tree and the
oracle."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from conftest import ROOT, load_golden

pytestmark = pytest.mark.gpu


def _parse_tree(lines):
    parent, frame, depth, excl, incl = [], [], [], [], []
    for ln in lines:
        _, p, f, d, e, i = ln.split()
        parent.append(int(p)); frame.append(int(f)); depth.append(int(d)); excl.append(int(e)); incl.append(int(i))
    return {"parent": np.array(parent, np.uint32), "frame": np.array(frame, np.uint32),
            "depth": np.array(depth, np.uint32), "excl": np.array(excl, np.uint64)[:, None],
            "incl": np.array(incl, np.uint64)[:, None]}


def test_plain_c_client(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc is not available")
    pkg = os.path.join(ROOT, "paper_2411_02797_amd")
    exe = str(tmp_path / "cct_c_example")
    subprocess.run(["gcc", "-std=c11", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include", "-I",
                    os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c_abi", "cct_c_example.c"),
                    "-L", pkg, "-lcct", "-L", "/opt/rocm/lib", "-lamdhip64", f"-Wl,-rpath,{pkg}",
                    "-Wl,-rpath,/opt/rocm/lib", "-o", exe], check=True)
    out = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    lines = out.stdout.splitlines()
    b = lines.index(next(ln for ln in lines if ln.startswith("BUILD")))
    m = lines.index(next(ln for ln in lines if ln.startswith("MERGE")))
    _, u1, d1 = lines[b].split()
    built = _parse_tree(lines[b + 1:b + 1 + int(u1)])
    _, u2, d2 = lines[m].split()
    merged = _parse_tree(lines[m + 1:m + 1 + int(u2)])
    o, f, w, want = load_golden("W1.txt")
    assert int(d1) == 5
    for k in ("parent", "frame", "depth", "excl", "incl"):
        assert np.array_equal(built[k], want[k]), k
    o2 = np.array([0, 2, 4]); f2 = np.array([1, 2, 4, 5], np.uint32); w2 = np.array([[4], [6]], np.uint64)
    want2 = oracle.build_tree(np.concatenate([o, o[-1] + o2[1:]]), np.concatenate([f, f2]), np.concatenate([w, w2]))
    assert int(d2) == 6
    for k in ("parent", "frame", "depth", "excl", "incl"):
        assert np.array_equal(merged[k], want2[k]), k
    q = lines[-1].split()
    assert q[0] == "Q"
    node = next(v for v in range(want2["parent"].size)
                if want2["depth"][v] == 2 and want2["frame"][v] == 2 and want2["frame"][want2["parent"][v]] == 1)
    assert (int(q[1]), int(q[2]), int(q[3]), int(q[4])) == (node, int(want2["incl"][node, 0]), -1, 0)
