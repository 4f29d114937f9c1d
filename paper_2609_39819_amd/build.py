"""Build ``libkvt.so`` (the C-ABI library) in-tree with hipcc for gfx950.

``python -m paper_2609_39819_amd.build`` compiles every source under
``csrc/`` into objects under ``_build/`` (in parallel), links
``paper_2609_39819_amd/libkvt.so`` next to this file, and builds the tests'
native caller of the C ABI, ``tests/kvt_run`` (from ``tests/kvt_run.cpp``).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libkvt.so")
RUNNER = os.path.join(ROOT, "tests", "kvt_run")   # a native (C++) caller of the C ABI, for the tests
ARCH = "gfx950"

# Packed fp32 VALU forms are kept out of device code (-packed-fp32-ops).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libkvt.so)")


def _compile(src: str, obj: str) -> None:
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
           "-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj]
    if src.endswith(".hip"):
        cmd[1:1] = DEVICE_FLAGS
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))
    objs = []
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        futs = []
        for f in srcs:
            obj = os.path.join(BUILD, f + ".o")
            objs.append(obj)
            futs.append(ex.submit(_compile, os.path.join(CSRC, f), obj))
        for fu in futs:
            fu.result()
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    # the native caller used by the tests: host code only, finds the library by rpath
    cmd = [hipcc(), "-O2", "-std=c++17", "-Wall", "-I", INCLUDE, RUNNER + ".cpp", "-o", RUNNER + ".tmp",
           "-L", PKG, "-lkvt", "-Wl,-rpath,$ORIGIN/../paper_2609_39819_amd"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build of {RUNNER} failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(RUNNER + ".tmp", RUNNER)
    if verbose:
        print(f"built {LIB} and {RUNNER}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
