"""CPU oracle for the HCCL collective semantics -- TEST INFRASTRUCTURE, not the product.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import this package. The GPU library never imports it, and it imports nothing of the GPU
library: the two share no code. The arithmetic lives in ``hccl_oracle.c`` (plain C, one
element and one contributor at a time); this module only builds it with gcc and marshals
numpy arrays through ctypes.

Semantics (paper, Section II-A-2 "Near Memory Compute" and Section III-B-2 "Data Path"):
BF16 / FP16 / FP32 buffers are reduced with FP32 arithmetic and re-quantised once to the
buffer type with round-to-nearest-even; INT32 sums wrap modulo 2^32. The contributors of an
element are folded in ascending rank order (``group=0``) or in the two-level order
(``group=L``: ascending inside each group of L consecutive ranks, FP32 partials, then
ascending over groups). Element data is passed as raw bits: ``uint16`` arrays for
bf16 / fp16, ``float32`` for fp32, ``int32`` for int32.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hccl_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

DTYPES = {"bf16": 0, "fp16": 1, "fp32": 2, "int32": 3}
OPS = {"sum": 0, "max": 1, "min": 2}
NP_STORAGE = {"bf16": np.uint16, "fp16": np.uint16, "fp32": np.float32, "int32": np.int32}

_lib = None

ORDERS = {"ascending": 0, "two_level": 1, "ring": 2, "halving": 3}


class OrderSpec(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("group", ctypes.c_int), ("shard", ctypes.c_size_t),
                ("requant", ctypes.c_int)]


def _order(order: str, group: int, shard: int, requant: bool) -> OrderSpec:
    return OrderSpec(ORDERS[order], int(group), int(shard), 1 if requant else 0)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math, no FP contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-Wextra", "-o", tmp, _SRC]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = _bind(ctypes.CDLL(_LIB))
    return _lib


def _bind(lib):
    """Declare the C signatures on a loaded oracle library."""
    vp, sz, i = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
    vpp = ctypes.POINTER(ctypes.c_void_p)
    szp = ctypes.POINTER(ctypes.c_size_t)
    lib.orc_bf16_to_f32.restype = ctypes.c_float
    lib.orc_bf16_to_f32.argtypes = [ctypes.c_uint16]
    lib.orc_f32_to_bf16.restype = ctypes.c_uint16
    lib.orc_f32_to_bf16.argtypes = [ctypes.c_float]
    lib.orc_f16_to_f32.restype = ctypes.c_float
    lib.orc_f16_to_f32.argtypes = [ctypes.c_uint16]
    lib.orc_f32_to_f16.restype = ctypes.c_uint16
    lib.orc_f32_to_f16.argtypes = [ctypes.c_float]
    for name in ("orc_f32_to_bf16_array", "orc_f32_to_f16_array", "orc_f16_to_f32_array"):
        getattr(lib, name).restype = None
        getattr(lib, name).argtypes = [vp, vp, sz]
    lib.orc_allreduce.restype = i
    lib.orc_allreduce.argtypes = [i, sz, i, i, i, vpp, vpp]
    lib.orc_reduce_scatter.restype = i
    lib.orc_reduce_scatter.argtypes = [i, sz, i, i, i, vpp, vpp]
    lib.orc_allgather.restype = i
    lib.orc_allgather.argtypes = [i, sz, sz, vpp, vpp]
    lib.orc_alltoallv.restype = i
    lib.orc_alltoallv.argtypes = [i, sz, vpp, szp, szp, vpp, szp, szp]
    i64p = ctypes.POINTER(ctypes.c_int64)
    lib.orc_alltoallv_dynamic.restype = i
    lib.orc_alltoallv_dynamic.argtypes = [i, sz, sz, vpp, sz, i64p, i64p, vpp, sz, i64p, i64p]
    lib.orc_allreduce_ordered.restype = i
    lib.orc_allreduce_ordered.argtypes = [i, sz, i, i, ctypes.POINTER(OrderSpec), vpp, vpp]
    lib.orc_reduce_scatter_ordered.restype = i
    lib.orc_reduce_scatter_ordered.argtypes = [i, sz, i, i, ctypes.POINTER(OrderSpec), vpp, vpp]
    return lib


class use_library:
    """Context manager that points this module at another build of the oracle source
    (the mutation tests compile deliberately broken copies and check the pins reject them)."""

    def __init__(self, path: str):
        self.path = path
        self.saved = None

    def __enter__(self):
        global _lib
        self.saved = _load()
        _lib = None
        lib = ctypes.CDLL(self.path)
        _lib = _bind(lib)
        return self

    def __exit__(self, *exc):
        global _lib
        _lib = self.saved
        return False


def _ptrs(arrays) -> ctypes.Array:
    return (ctypes.c_void_p * len(arrays))(*[a.ctypes.data for a in arrays])


def _sizes(a) -> ctypes.Array:
    flat = np.ascontiguousarray(a, dtype=np.uint64).reshape(-1)
    return (ctypes.c_size_t * flat.size)(*[int(v) for v in flat])


def _rows(x: np.ndarray, dtype: str):
    want = NP_STORAGE[dtype]
    if x.dtype != want:
        raise TypeError(f"{dtype} data must be passed as {np.dtype(want).name} bits, got {x.dtype}")
    return [np.ascontiguousarray(x[r]) for r in range(x.shape[0])]


# --------------------------------------------------------------------------- conversions
def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().orc_f32_to_bf16_array(x.ctypes.data, out.ctypes.data, x.size)
    return out


def bf16_to_f32(h: np.ndarray) -> np.ndarray:
    h = np.ascontiguousarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32)


def f32_to_f16(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().orc_f32_to_f16_array(x.ctypes.data, out.ctypes.data, x.size)
    return out


def f16_to_f32(h: np.ndarray) -> np.ndarray:
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.empty(h.shape, dtype=np.float32)
    _load().orc_f16_to_f32_array(h.ctypes.data, out.ctypes.data, h.size)
    return out


# --------------------------------------------------------------------------- collectives
def allreduce(x: np.ndarray, dtype: str, op: str = "sum", group: int = 0) -> np.ndarray:
    """x: (P, N) element bits per rank -> (P, N) outputs (every row the same)."""
    P, N = x.shape
    rows = _rows(x, dtype)
    out = [np.empty(N, dtype=NP_STORAGE[dtype]) for _ in range(P)]
    rc = _load().orc_allreduce(P, N, DTYPES[dtype], OPS[op], group, _ptrs(rows), _ptrs(out))
    if rc != 0:
        raise ValueError(f"orc_allreduce rejected its arguments (rc={rc})")
    return np.stack(out) if P else np.empty((0, N), NP_STORAGE[dtype])


def reduce_scatter(x: np.ndarray, dtype: str, op: str = "sum", group: int = 0) -> np.ndarray:
    """x: (P, P*M) element bits per rank -> (P, M): row c is the reduction of block c."""
    P, total = x.shape
    if total % P:
        raise ValueError("reduce_scatter input length must be a multiple of P")
    M = total // P
    rows = _rows(x, dtype)
    out = [np.empty(M, dtype=NP_STORAGE[dtype]) for _ in range(P)]
    rc = _load().orc_reduce_scatter(P, M, DTYPES[dtype], OPS[op], group, _ptrs(rows), _ptrs(out))
    if rc != 0:
        raise ValueError(f"orc_reduce_scatter rejected its arguments (rc={rc})")
    return np.stack(out)


def allreduce_ordered(x: np.ndarray, dtype: str, order: str = "ascending", op: str = "sum", group: int = 0,
                      shard: int = 0, requant: bool = False) -> np.ndarray:
    """All-reduce in an explicit fold order (see hccl_oracle.h): "ascending", "two_level"
    (group), "ring" (rotated per shard of `shard` elements), "halving"; requant rounds every
    partial to the buffer type."""
    P, N = x.shape
    rows = _rows(x, dtype)
    out = [np.empty(N, dtype=NP_STORAGE[dtype]) for _ in range(P)]
    spec = _order(order, group, shard, requant)
    rc = _load().orc_allreduce_ordered(P, N, DTYPES[dtype], OPS[op], ctypes.byref(spec), _ptrs(rows), _ptrs(out))
    if rc != 0:
        raise ValueError(f"orc_allreduce_ordered rejected its arguments (rc={rc})")
    return np.stack(out)


def reduce_scatter_ordered(x: np.ndarray, dtype: str, order: str = "ascending", op: str = "sum",
                           group: int = 0, requant: bool = False) -> np.ndarray:
    """Reduce-scatter in an explicit fold order; for "ring", block c is folded starting at
    contributor c+1."""
    P, total = x.shape
    if total % P:
        raise ValueError("reduce_scatter input length must be a multiple of P")
    M = total // P
    rows = _rows(x, dtype)
    out = [np.empty(M, dtype=NP_STORAGE[dtype]) for _ in range(P)]
    spec = _order(order, group, 0, requant)
    rc = _load().orc_reduce_scatter_ordered(P, M, DTYPES[dtype], OPS[op], ctypes.byref(spec), _ptrs(rows),
                                            _ptrs(out))
    if rc != 0:
        raise ValueError(f"orc_reduce_scatter_ordered rejected its arguments (rc={rc})")
    return np.stack(out)


def allgather(x: np.ndarray) -> np.ndarray:
    """x: (P, M) per-rank blocks (any element type) -> (P, P*M)."""
    P, M = x.shape
    rows = [np.ascontiguousarray(x[r]) for r in range(P)]
    out = [np.empty(P * M, dtype=x.dtype) for _ in range(P)]
    rc = _load().orc_allgather(P, M, x.dtype.itemsize, _ptrs(rows), _ptrs(out))
    if rc != 0:
        raise ValueError(f"orc_allgather rejected its arguments (rc={rc})")
    return np.stack(out)


def alltoallv(send: list, sendcounts, sdispls, recv: list, recvcounts, rdispls) -> list:
    """AllToAllv over P per-rank 1-D arrays. ``recv`` arrays are updated in place (bytes
    outside every written range keep their value) and returned. Counts and displacements
    are (P, P) element arrays: send side indexed [src, dst], receive side [dst, src]."""
    P = len(send)
    if len(recv) != P:
        raise ValueError("send and recv must list the same number of ranks")
    es = send[0].dtype.itemsize
    for a in list(send) + list(recv):
        if a.dtype.itemsize != es or not a.flags["C_CONTIGUOUS"]:
            raise ValueError("all buffers must be contiguous and share one element size")
    rc = _load().orc_alltoallv(P, es, _ptrs(send), _sizes(sendcounts), _sizes(sdispls),
                               _ptrs(recv), _sizes(recvcounts), _sizes(rdispls))
    if rc != 0:
        raise ValueError(f"orc_alltoallv rejected its arguments (rc={rc})")
    return recv


def _i64(a):
    if a is None:
        return None
    flat = np.ascontiguousarray(a, dtype=np.int64).reshape(-1)
    return (ctypes.c_int64 * flat.size)(*[int(v) for v in flat])


def alltoallv_dynamic(send: list, counts, recv: list, row_elems: int, send_cap: int, recv_cap: int,
                      sdispls=None, rdispls=None):
    """AllToAllvDynamic (see hccl_oracle.h): ``counts`` (P, P) rows indexed [src, dst];
    ``sdispls`` [src, dst] and ``rdispls`` [dst, src] row offsets, None = packed. ``send[s]``
    holds ``send_cap`` rows and ``recv[d]`` ``recv_cap`` rows of ``row_elems`` elements.
    Returns (accepted, recvcounts): ``recv`` is updated in place only when the layout is
    accepted; recvcounts (P, P) [dst, src] is the transposed count matrix either way."""
    P = len(send)
    if len(recv) != P:
        raise ValueError("send and recv must list the same number of ranks")
    es = send[0].dtype.itemsize
    for a in send:
        if a.size != send_cap * row_elems or a.dtype.itemsize != es or not a.flags["C_CONTIGUOUS"]:
            raise ValueError("every send buffer must be contiguous and hold send_cap rows")
    for a in recv:
        if a.size != recv_cap * row_elems or a.dtype.itemsize != es or not a.flags["C_CONTIGUOUS"]:
            raise ValueError("every receive buffer must be contiguous and hold recv_cap rows")
    rc_out = (ctypes.c_int64 * (P * P))()
    rc = _load().orc_alltoallv_dynamic(P, es, int(row_elems), _ptrs(send), int(send_cap), _i64(counts),
                                       _i64(sdispls), _ptrs(recv), int(recv_cap), _i64(rdispls), rc_out)
    if rc == -1:
        raise ValueError("orc_alltoallv_dynamic rejected its arguments")
    return rc == 0, np.array(rc_out[:], dtype=np.int64).reshape(P, P)
