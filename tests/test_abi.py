"""The C-ABI library loads on the CPU and exports every entry point include/cct.h
declares (no compute calls: there is no GPU here)."""
import ctypes
import os
import re
import shutil
import subprocess

import pytest

import paper_2411_02797_amd as cct

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "cct.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cct_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_symbols()
    for required in ("cct_build", "cct_merge", "cct_query", "cct_export", "cct_free", "cct_info"):
        assert required in names


def test_header_is_plain_c_and_links(tmp_path):
    # the plain C client of the GPU tests compiles as C11 with every warning an error and
    # links against libcct.so and the HIP runtime (it is not run: there is no GPU here)
    if shutil.which("gcc") is None or not os.path.isdir("/opt/rocm/include"):
        pytest.skip("gcc or the HIP headers are not available")
    pkg = os.path.dirname(cct.library_path())
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I",
                    "/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_abi", "cct_c_example.c"), "-L", pkg, "-lcct", "-L",
                    "/opt/rocm/lib", "-lamdhip64", "-o", str(tmp_path / "cct_c_example")], check=True)
    assert os.path.exists(tmp_path / "cct_c_example")


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(cct.library_path())
    for name in declared_symbols():
        assert hasattr(lib, name), f"libcct.so does not export {name}"
    assert set(declared_symbols()) == set(cct.EXPORTED_SYMBOLS)


def test_null_arguments_rejected_without_gpu_work():
    lib = cct.load_library()
    out = ctypes.c_void_p()
    assert lib.cct_build(None, None, ctypes.byref(out)) == -1
    assert b"NULL" in lib.cct_last_error()
    p = cct._Paths(3, 0, 0, 8, None, None)  # n_metrics 0
    assert lib.cct_build(ctypes.byref(p), None, ctypes.byref(out)) == -1
    p = cct._Paths(3, 0, 9, 8, None, None)  # n_metrics 9
    assert lib.cct_build(ctypes.byref(p), None, ctypes.byref(out)) == -1
    p = cct._Paths(-1, 0, 1, 8, None, None)
    assert lib.cct_build(ctypes.byref(p), None, ctypes.byref(out)) == -1
    p = cct._Paths(2**31, 0, 1, 8, None, 8)
    assert lib.cct_build(ctypes.byref(p), None, ctypes.byref(out)) == -5
    assert lib.cct_merge(None, ctypes.byref(p), None) == -1
    lib.cct_free(None)  # NULL-safe


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(cct, "_LIB_PATH", str(tmp_path / "absent.so"))
    monkeypatch.setattr(cct, "_lib", None)
    with pytest.raises(ImportError):
        cct.load_library()


def test_noalloc_filter_rejects_null_arguments_without_gpu_work():
    lib = cct.load_library()
    k = ctypes.c_int64(-3)
    spec = cct._FilterSpec(0, 0, 0, 0, 0, 1, 1, 1, 0)
    assert lib.cct_filter_noalloc(None, ctypes.byref(spec), None, 0, None, ctypes.byref(k)) == -1
    assert k.value == -3
    assert b"NULL" in lib.cct_last_error()
