"""Builds libhccl.so in-tree for gfx950.

Host-only sources (the descriptor compiler and validator) are compiled with g++; the
executor and the C ABI (which calls the HIP runtime and launches kernels) with hipcc for
gfx950. Packed FP32 instructions are disabled for all device code.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libhccl.so")
OBJDIR = os.path.join(PKG, "_build")
ARCH = "gfx950"

HOST_SOURCES = ["compiler.cpp", "validate.cpp"]
HIP_SOURCES = ["executor.hip", "api.cpp"]

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
GXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-Wno-unused-parameter"]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def _compile(src: str) -> str:
    path = os.path.join(CSRC, src)
    obj = os.path.join(OBJDIR, src + ".o")
    inc = ["-I", INCLUDE, "-I", CSRC]
    if src in HOST_SOURCES:
        cmd = ["g++", *GXX_FLAGS, *inc, "-c", path, "-o", obj]
    else:
        cmd = [_hipcc(), *HIPCC_FLAGS, *inc, "-x", "hip", "-c", path, "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


BENCH_STREAM_SRC = os.path.join(ROOT, "bench_stream.hip")
BENCH_STREAM_LIB = os.path.join(LIBDIR, "libbench_stream.so")


def build_bench_stream() -> str:
    """The STREAM-style reference kernels bench.py times beside the collectives (not part of
    libhccl.so)."""
    os.makedirs(LIBDIR, exist_ok=True)
    tmp = BENCH_STREAM_LIB + ".tmp"
    cmd = [_hipcc(), *HIPCC_FLAGS, "-shared", "-x", "hip", BENCH_STREAM_SRC, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, BENCH_STREAM_LIB)
    return BENCH_STREAM_LIB


def build() -> str:
    """Compiles every source and links lib/libhccl.so. Always rebuilds."""
    os.makedirs(OBJDIR, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(_compile, HOST_SOURCES + HIP_SOURCES))
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
