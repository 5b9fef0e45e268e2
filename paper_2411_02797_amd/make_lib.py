"""Compile libcct.so (HIP kernels + host runtime) for gfx950 with hipcc, in place."""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libcct.so")
# the read-bandwidth probe the bench reports beside the tree-building kernels (not part
# of the library's API)
READBW_SRC = "readbw.hip"
READBW_OUT = os.path.join(HERE, "libcct_readbw.so")
SOURCES = ["ingest.hip", "canon.hip", "trie.hip", "query.hip", "activity.hip", "bottomup.hip", "filter.hip", "stats.hip", "runtime.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         "-I", os.path.join(os.path.dirname(HERE), "include"),
         # packed FP32 instructions are kept out of every code object
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build(verbose: bool = False, jobs: int = 4) -> str:
    bdir = os.path.join(os.path.dirname(HERE), "_build")
    os.makedirs(bdir, exist_ok=True)
    objs = []

    def compile_one(src):
        obj = os.path.join(bdir, os.path.splitext(src)[0] + ".o")
        cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
        warn = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip())
        if verbose and warn:
            print(warn)
        return obj

    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True, capture_output=not verbose)
    os.replace(tmp, OUT)
    tmp = READBW_OUT + ".tmp"
    cmd = [HIPCC, *FLAGS, "-shared", os.path.join(CSRC, READBW_SRC), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {READBW_SRC}:\n{r.stderr}")
    os.replace(tmp, READBW_OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
