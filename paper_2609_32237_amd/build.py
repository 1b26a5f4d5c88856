"""Build libmi355fft.so (HIP, gfx950) in-tree with hipcc.

Every translation unit is compiled for gfx950 only, with packed-FP32 VALU
instructions disabled (``-target-feature -packed-fp32-ops``); the host pass
of hipcc warns that it does not know that feature, which is harmless.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmi355fft.so")
OBJ_DIR = os.path.join(PKG, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
] + [f"-D{d}" for d in os.environ.get("MI355FFT_DEFINES", "").split() if d]
SOURCES = ["fft_small.hip", "fft_n1024.hip", "fft_n2048.hip", "fft_n4096.hip", "fft_n8192.hip", "fft_n16384.hip",
           "noalloc.hip", "runtime.cpp"]
# the memory-ceiling kernels of the benchmark: a library of their own, which
# the FFT library neither links nor calls
MEMBENCH_SOURCES = ["membench.hip"]
MEMBENCH_LIB = os.path.join(PKG, "libmi355membench.so")


def _compile(src: str) -> str:
    obj = os.path.join(OBJ_DIR, os.path.splitext(src)[0] + ".o")
    path = os.path.join(CSRC, src)
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC, *COMMON, *lang, "-c", path, "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (res.stderr or "").splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        print(err, file=sys.stderr)
    return obj


def _link(objs, lib):
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    os.replace(tmp, lib)


def build(jobs: int | None = None, verbose: bool = True) -> str:
    """Compile every source and link the shared libraries; returns the FFT
    library's path."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    srcs = SOURCES + MEMBENCH_SOURCES
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 1)), 8)
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, srcs))
    _link(objs[:len(SOURCES)], LIB)
    _link(objs[len(SOURCES):], MEMBENCH_LIB)
    if verbose:
        print(f"built {LIB}")
        print(f"built {MEMBENCH_LIB}")
    return LIB


if __name__ == "__main__":
    build()
