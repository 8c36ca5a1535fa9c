"""Builds libhccl.so in-tree for gfx950.

Host-only sources (the descriptor compiler and validator) are compiled with g++; the
executor and the C ABI (which calls the HIP runtime and launches kernels) with hipcc for
gfx950. Packed FP32 instructions are disabled for all device code, and every gfx950 code
object built here is disassembled and rejected if it holds one anyway: the compiler still
emits `v_pk_mov_b32` for some vector shuffles with the feature off.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import tempfile

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


# packed FP32 arithmetic and the packed 32-bit move of the same instruction group
PACKED_FP32 = re.compile(r"\bv_pk_(?:add|mul|fma)_f32\b|\bv_pk_mov_b32\b")


def _llvm_tool(name: str) -> str:
    for cand in (os.path.join("/opt/rocm/llvm/bin", name), shutil.which(name)):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError(f"{name} not found: the device code cannot be checked")


def check_device_code(path: str) -> None:
    """Disassembles the gfx950 code object embedded in `path` (an object file or shared library
    built here) and raises if it holds a packed FP32 instruction."""
    with tempfile.TemporaryDirectory() as tmp:
        fatbin, co = os.path.join(tmp, "fatbin"), os.path.join(tmp, "device.co")
        steps = [
            [_llvm_tool("llvm-objcopy"), f"--dump-section=.hip_fatbin={fatbin}", path, os.path.join(tmp, "host")],
            [_llvm_tool("clang-offload-bundler"), "--type=o", f"--targets=hipv4-amdgcn-amd-amdhsa--{ARCH}",
             f"--input={fatbin}", f"--output={co}", "--unbundle"],
        ]
        for cmd in steps:
            res = subprocess.run(cmd, capture_output=True, text=True)
            if res.returncode != 0:
                raise RuntimeError(f"device code check failed: {' '.join(cmd)}\n{res.stderr}")
        res = subprocess.run([_llvm_tool("llvm-objdump"), "-d", f"--mcpu={ARCH}", co], capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"device code check failed: llvm-objdump\n{res.stderr}")
        found = sorted(set(PACKED_FP32.findall(res.stdout)))
        if found:
            raise RuntimeError(f"{path}: packed FP32 instructions in the device code: {', '.join(found)}")


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
    check_device_code(tmp)
    os.replace(tmp, BENCH_STREAM_LIB)
    return BENCH_STREAM_LIB


def build() -> str:
    """Compiles every source and links lib/libhccl.so. Always rebuilds."""
    os.makedirs(OBJDIR, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(_compile, HOST_SOURCES + HIP_SOURCES))
    check_device_code(os.path.join(OBJDIR, "executor.hip.o"))
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
