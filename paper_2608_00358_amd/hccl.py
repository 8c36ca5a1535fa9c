"""ctypes binding of libhccl.so: argument marshalling only.

Every function here has the name of the C entry point it calls and turns Python arguments
(torch tensors or raw device addresses, strings for enums) into the C arguments. All
collective work runs in the HIP library; if the library is not built, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "lib", "libhccl.so")

DTYPES = {"bf16": 0, "fp16": 1, "fp32": 2, "int32": 3}
OPS = {"sum": 0, "max": 1, "min": 2}
ALGOS = {"auto": 0, "direct": 1, "ring": 2, "two_level": 3, "rhd": 4}
ORDERS = {"ascending": 0, "ring": 1, "halving": 2}
PHASES = {"auto": 0, "one": 1, "levels": 2}
RESULTS = {0: "hcclSuccess", 1: "hcclInvalidArgument", 2: "hcclUnsupported", 3: "hcclHipError",
           4: "hcclOutOfMemory", 5: "hcclTimeout", 6: "hcclInternalError"}
NO_DEVICE = -1
MAX_RANKS = 64

# Every symbol include/hccl.h declares.
EXPORTS = [
    "hccl_config_init", "hccl_comm_create", "hccl_comm_destroy", "hccl_comm_set_config",
    "hccl_allreduce", "hccl_reduce_scatter", "hccl_allgather", "hccl_alltoallv",
    "hccl_get_last_error", "hccl_result_string", "hccl_get_async_error", "hccl_comm_last_program",
    "hccl_group_start", "hccl_group_end", "hccl_alltoallv_dynamic", "hccl_set_trigger",
    "hccl_resident_start", "hccl_resident_stop", "hccl_resident_wait", "hccl_resident_last_seq",
    "hccl_allreduce_noalloc", "hccl_comm_trace", "hccl_comm_program_image",
]
CMPS = {"eq": 0, "ne": 1, "ge": 2, "gt": 3, "le": 4, "lt": 5}


class HcclError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{RESULTS.get(code, code)}: {message}")
        self.code = code


class hcclConfig_t(ctypes.Structure):
    _fields_ = [
        ("algo", ctypes.c_int32), ("group_size", ctypes.c_int32), ("chunk_bytes", ctypes.c_uint64),
        ("fuse", ctypes.c_int32), ("max_workers", ctypes.c_int32), ("tile_bytes", ctypes.c_uint32),
        ("timeout_ms", ctypes.c_uint32), ("validate", ctypes.c_int32), ("order", ctypes.c_int32),
        ("requantize", ctypes.c_int32), ("trace", ctypes.c_int32), ("phases", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


class hcclTrigger_t(ctypes.Structure):
    _fields_ = [
        ("wait_addr", ctypes.c_void_p), ("wait_value", ctypes.c_uint64), ("wait_cmp", ctypes.c_int32),
        ("reserved", ctypes.c_int32), ("done_addr", ctypes.c_void_p), ("done_value", ctypes.c_uint64),
    ]


class hcclProgramInfo_t(ctypes.Structure):
    _fields_ = [
        ("collective", ctypes.c_int32), ("algo", ctypes.c_int32), ("fused", ctypes.c_int32),
        ("cache_hit", ctypes.c_int32), ("num_descs", ctypes.c_uint32), ("num_tiles", ctypes.c_uint32),
        ("num_deps", ctypes.c_uint32), ("num_operands", ctypes.c_uint32), ("workers", ctypes.c_uint32),
        ("max_srcs", ctypes.c_uint32), ("inline_launch", ctypes.c_uint32), ("tickets", ctypes.c_uint32),
        ("bytes_read", ctypes.c_uint64), ("bytes_written", ctypes.c_uint64),
        ("scratch_bytes", ctypes.c_uint64), ("program_bytes", ctypes.c_uint64), ("compile_us", ctypes.c_double),
        ("step_tile_min", ctypes.c_uint32), ("step_tile_max", ctypes.c_uint32),
        ("num_phases", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
    ]


class hcclTileTrace_t(ctypes.Structure):
    _fields_ = [
        ("start", ctypes.c_uint64), ("ready", ctypes.c_uint32), ("done", ctypes.c_uint32),
        ("wave", ctypes.c_uint32), ("where", ctypes.c_uint32), ("reserved", ctypes.c_uint64),
    ]


_lib = None


def load(path: str = LIB_PATH):
    """Loads libhccl.so (built by ``__graft_entry__.build()``); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run __graft_entry__.build() first "
                           "(the collectives exist only as HIP code)")
    lib = ctypes.CDLL(path)
    vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
    vpp = ctypes.POINTER(ctypes.c_void_p)
    szp = ctypes.POINTER(ctypes.c_size_t)
    res = ctypes.c_int
    lib.hccl_config_init.argtypes = [ctypes.POINTER(hcclConfig_t)]
    lib.hccl_comm_create.argtypes = [i32, i32, ctypes.POINTER(hcclConfig_t), ctypes.POINTER(vp)]
    lib.hccl_comm_destroy.argtypes = [vp]
    lib.hccl_comm_set_config.argtypes = [vp, ctypes.POINTER(hcclConfig_t)]
    lib.hccl_allreduce.argtypes = [vp, vpp, vpp, sz, i32, i32, vp]
    lib.hccl_allreduce_noalloc.argtypes = [vp, vpp, vpp, sz, i32, i32, vp]
    lib.hccl_reduce_scatter.argtypes = [vp, vpp, vpp, sz, i32, i32, vp]
    lib.hccl_allgather.argtypes = [vp, vpp, vpp, sz, i32, vp]
    lib.hccl_alltoallv.argtypes = [vp, vpp, szp, szp, vpp, szp, szp, i32, vp]
    lib.hccl_alltoallv_dynamic.argtypes = [vp, vpp, vp, vp, vpp, vp, vp, sz, sz, sz, i32, vp]
    lib.hccl_set_trigger.argtypes = [vp, ctypes.POINTER(hcclTrigger_t)]
    lib.hccl_get_last_error.argtypes = []
    lib.hccl_get_last_error.restype = ctypes.c_char_p
    lib.hccl_result_string.argtypes = [i32]
    lib.hccl_result_string.restype = ctypes.c_char_p
    lib.hccl_get_async_error.argtypes = [vp]
    lib.hccl_comm_last_program.argtypes = [vp, ctypes.POINTER(hcclProgramInfo_t)]
    lib.hccl_comm_program_image.argtypes = [vp, vp, sz, ctypes.POINTER(ctypes.c_size_t)]
    lib.hccl_comm_trace.argtypes = [vp, ctypes.POINTER(hcclTileTrace_t), sz, ctypes.POINTER(ctypes.c_size_t),
                                    ctypes.POINTER(ctypes.c_uint64)]
    lib.hccl_group_start.argtypes = [vp]
    lib.hccl_group_end.argtypes = [vp]
    lib.hccl_resident_start.argtypes = [vp, ctypes.c_uint32, ctypes.c_uint32]
    lib.hccl_resident_stop.argtypes = [vp]
    lib.hccl_resident_wait.argtypes = [vp, ctypes.c_uint64, ctypes.c_uint32]
    lib.hccl_resident_last_seq.argtypes = [vp, ctypes.POINTER(ctypes.c_uint64)]
    for name in EXPORTS:
        if name not in ("hccl_get_last_error", "hccl_result_string"):
            getattr(lib, name).restype = res
    _lib = lib
    return lib


def _check(rc: int):
    if rc != 0:
        raise HcclError(rc, load().hccl_get_last_error().decode())


def _addr(x) -> int:
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _addr_or_null(x) -> Optional[int]:
    return None if x is None else _addr(x)


def _ptr_array(bufs: Sequence) -> ctypes.Array:
    return (ctypes.c_void_p * len(bufs))(*[_addr(b) for b in bufs])


def _size_array(a) -> ctypes.Array:
    flat = [int(v) for v in (a.reshape(-1).tolist() if hasattr(a, "reshape") else a)]
    return (ctypes.c_size_t * len(flat))(*flat)


def _dtype_code(dtype) -> int:
    if isinstance(dtype, str):
        return DTYPES[dtype]
    if isinstance(dtype, int):
        return dtype
    import torch

    table = {torch.bfloat16: 0, torch.float16: 1, torch.float32: 2, torch.int32: 3}
    if dtype not in table:
        raise TypeError(f"unsupported element type {dtype}")
    return table[dtype]


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch

        if torch.cuda.is_available():
            return torch.cuda.current_stream().cuda_stream
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def hccl_config_init(**kw) -> hcclConfig_t:
    cfg = hcclConfig_t()
    _check(load().hccl_config_init(ctypes.byref(cfg)))
    for k, v in kw.items():
        if k == "algo" and isinstance(v, str):
            v = ALGOS[v]
        if k == "order" and isinstance(v, str):
            v = ORDERS[v]
        if k == "phases" and isinstance(v, str):
            v = PHASES[v]
        setattr(cfg, k, int(v))
    return cfg


def hccl_comm_create(nranks: int, device: int = 0, cfg: Optional[hcclConfig_t] = None) -> ctypes.c_void_p:
    comm = ctypes.c_void_p()
    _check(load().hccl_comm_create(nranks, device, ctypes.byref(cfg) if cfg is not None else None,
                                   ctypes.byref(comm)))
    return comm


def hccl_comm_destroy(comm) -> None:
    _check(load().hccl_comm_destroy(comm))


def hccl_comm_set_config(comm, cfg: hcclConfig_t) -> None:
    _check(load().hccl_comm_set_config(comm, ctypes.byref(cfg)))


def hccl_allreduce(comm, sendbufs, recvbufs, count: int, dtype, op: str = "sum", stream=None) -> None:
    _check(load().hccl_allreduce(comm, _ptr_array(sendbufs), _ptr_array(recvbufs), count, _dtype_code(dtype),
                                 OPS[op], _stream_handle(stream)))


def hccl_allreduce_noalloc(comm, sendbufs, recvbufs, count: int, dtype, op: str = "sum", stream=None) -> None:
    _check(load().hccl_allreduce_noalloc(comm, _ptr_array(sendbufs), _ptr_array(recvbufs), count, _dtype_code(dtype),
                                         OPS[op], _stream_handle(stream)))


def hccl_reduce_scatter(comm, sendbufs, recvbufs, recvcount: int, dtype, op: str = "sum", stream=None) -> None:
    _check(load().hccl_reduce_scatter(comm, _ptr_array(sendbufs), _ptr_array(recvbufs), recvcount,
                                      _dtype_code(dtype), OPS[op], _stream_handle(stream)))


def hccl_allgather(comm, sendbufs, recvbufs, sendcount: int, dtype, stream=None) -> None:
    _check(load().hccl_allgather(comm, _ptr_array(sendbufs), _ptr_array(recvbufs), sendcount,
                                 _dtype_code(dtype), _stream_handle(stream)))


def hccl_alltoallv(comm, sendbufs, sendcounts, sdispls, recvbufs, recvcounts, rdispls, dtype, stream=None) -> None:
    _check(load().hccl_alltoallv(comm, _ptr_array(sendbufs), _size_array(sendcounts), _size_array(sdispls),
                                 _ptr_array(recvbufs), _size_array(recvcounts), _size_array(rdispls),
                                 _dtype_code(dtype), _stream_handle(stream)))


def hccl_alltoallv_dynamic(comm, sendbufs, sendcounts, sdispls, recvbufs, recvcounts, rdispls, row_elems: int,
                           send_capacity: int, recv_capacity: int, dtype, stream=None) -> None:
    """Counts and offsets are device int64 arrays (tensors or addresses); sdispls, rdispls and
    recvcounts may be None."""
    _check(load().hccl_alltoallv_dynamic(comm, _ptr_array(sendbufs), _addr_or_null(sendcounts), _addr_or_null(sdispls),
                                         _ptr_array(recvbufs), _addr_or_null(recvcounts), _addr_or_null(rdispls),
                                         row_elems, send_capacity, recv_capacity, _dtype_code(dtype),
                                         _stream_handle(stream)))


def hccl_set_trigger(comm, wait=None, done=None) -> None:
    """Trigger for the next work packet: ``wait`` = (word, cmp, value) with cmp in CMPS,
    ``done`` = (word, value); words are device int64 tensors or addresses. Both None clears."""
    if wait is None and done is None:
        _check(load().hccl_set_trigger(comm, None))
        return
    t = hcclTrigger_t()
    if wait is not None:
        word, cmp, value = wait
        t.wait_addr, t.wait_cmp, t.wait_value = _addr(word), CMPS[cmp] if isinstance(cmp, str) else int(cmp), value
    if done is not None:
        word, value = done
        t.done_addr, t.done_value = _addr(word), value
    _check(load().hccl_set_trigger(comm, ctypes.byref(t)))


def hccl_group_start(comm) -> None:
    _check(load().hccl_group_start(comm))


def hccl_group_end(comm) -> None:
    _check(load().hccl_group_end(comm))


def hccl_get_last_error() -> str:
    return load().hccl_get_last_error().decode()


def hccl_result_string(code: int) -> str:
    return load().hccl_result_string(code).decode()


def hccl_get_async_error(comm) -> int:
    """Returns the result code (0 = no device-side error since the last call)."""
    return int(load().hccl_get_async_error(comm))


def hccl_resident_start(comm, blocks: int = 0, idle_ms: int = 0) -> None:
    _check(load().hccl_resident_start(comm, blocks, idle_ms))


def hccl_resident_stop(comm) -> None:
    _check(load().hccl_resident_stop(comm))


def hccl_resident_wait(comm, seq: int = 0, timeout_ms: int = 0) -> None:
    _check(load().hccl_resident_wait(comm, seq, timeout_ms))


def hccl_resident_last_seq(comm) -> int:
    out = ctypes.c_uint64(0)
    _check(load().hccl_resident_last_seq(comm, ctypes.byref(out)))
    return int(out.value)


def hccl_comm_last_program(comm) -> dict:
    info = hcclProgramInfo_t()
    _check(load().hccl_comm_last_program(comm, ctypes.byref(info)))
    return {name: getattr(info, name) for name, _ in hcclProgramInfo_t._fields_}


def hccl_comm_program_image(comm) -> bytes:
    """The packed image of the communicator's last program (b"" if none)."""
    lib = load()
    n = ctypes.c_size_t(0)
    _check(lib.hccl_comm_program_image(comm, None, 0, ctypes.byref(n)))
    buf = ctypes.create_string_buffer(max(1, n.value))
    _check(lib.hccl_comm_program_image(comm, buf, n.value, ctypes.byref(n)))
    return buf.raw[: n.value]


def hccl_comm_trace(comm):
    """Records of the last traced launch as a numpy structured array (fields start, ready, done,
    wave, where; times in wall-clock ticks) and the clock rate in kHz."""
    import numpy as np

    lib = load()
    n = ctypes.c_size_t(0)
    khz = ctypes.c_uint64(0)
    _check(lib.hccl_comm_trace(comm, None, 0, ctypes.byref(n), ctypes.byref(khz)))
    buf = (hcclTileTrace_t * max(1, n.value))()
    _check(lib.hccl_comm_trace(comm, buf, n.value, ctypes.byref(n), ctypes.byref(khz)))
    dt = np.dtype([("start", np.uint64), ("ready", np.uint32), ("done", np.uint32), ("wave", np.uint32),
                   ("where", np.uint32), ("reserved", np.uint64)])
    arr = np.frombuffer(bytes(buf), dtype=dt, count=n.value).copy()
    return arr, int(khz.value)


def _bound(fn, *args):
    def call():
        _check(fn(*args))

    return call


class Comm:
    """Convenience owner of one communicator; methods take lists of torch tensors."""

    def __init__(self, nranks: int, device: int = 0, **cfg):
        self.nranks = nranks
        self.device = device
        self.cfg = hccl_config_init(**cfg)
        self.handle = hccl_comm_create(nranks, device, self.cfg)

    def close(self):
        if self.handle is not None:
            hccl_comm_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
        return False

    def set_config(self, **cfg):
        self.cfg = hccl_config_init(**cfg)
        hccl_comm_set_config(self.handle, self.cfg)

    def allreduce(self, send, recv, op="sum", stream=None):
        hccl_allreduce(self.handle, send, recv, send[0].numel(), send[0].dtype, op, stream)

    def allreduce_noalloc(self, send, recv, op="sum", stream=None):
        hccl_allreduce_noalloc(self.handle, send, recv, send[0].numel(), send[0].dtype, op, stream)

    def reduce_scatter(self, send, recv, op="sum", stream=None):
        hccl_reduce_scatter(self.handle, send, recv, recv[0].numel(), send[0].dtype, op, stream)

    def allgather(self, send, recv, stream=None):
        hccl_allgather(self.handle, send, recv, send[0].numel(), send[0].dtype, stream)

    def alltoallv(self, send, sendcounts, sdispls, recv, recvcounts, rdispls, stream=None):
        hccl_alltoallv(self.handle, send, sendcounts, sdispls, recv, recvcounts, rdispls, send[0].dtype, stream)

    @staticmethod
    def _capacity(bufs, row_elems):
        n = bufs[0].numel()
        if any(b.numel() != n for b in bufs) or n % row_elems:
            raise ValueError("buffers must share one size, a whole number of rows")
        return n // row_elems

    def alltoallv_dynamic(self, send, counts, recv, row_elems, sdispls=None, rdispls=None, recvcounts=None,
                          stream=None):
        """AllToAllvDynamic: ``counts`` (and the optional offsets / received-count output) are
        int64 device tensors of P*P rows; capacities are the buffers' sizes in rows."""
        hccl_alltoallv_dynamic(self.handle, send, counts, sdispls, recv, recvcounts, rdispls, row_elems,
                               self._capacity(send, row_elems), self._capacity(recv, row_elems), send[0].dtype,
                               stream)

    # The bind_* methods marshal the arguments once and return a no-argument callable that
    # enqueues the collective: for loops that reuse the same buffers, where per-call ctypes
    # marshalling would otherwise cost more than a small collective itself.
    def bind_allreduce(self, send, recv, op="sum", stream=None):
        return _bound(load().hccl_allreduce, self.handle, _ptr_array(send), _ptr_array(recv), send[0].numel(),
                      _dtype_code(send[0].dtype), OPS[op], _stream_handle(stream))

    def bind_reduce_scatter(self, send, recv, op="sum", stream=None):
        return _bound(load().hccl_reduce_scatter, self.handle, _ptr_array(send), _ptr_array(recv), recv[0].numel(),
                      _dtype_code(send[0].dtype), OPS[op], _stream_handle(stream))

    def bind_allgather(self, send, recv, stream=None):
        return _bound(load().hccl_allgather, self.handle, _ptr_array(send), _ptr_array(recv), send[0].numel(),
                      _dtype_code(send[0].dtype), _stream_handle(stream))

    def bind_alltoallv(self, send, sendcounts, sdispls, recv, recvcounts, rdispls, stream=None):
        return _bound(load().hccl_alltoallv, self.handle, _ptr_array(send), _size_array(sendcounts),
                      _size_array(sdispls), _ptr_array(recv), _size_array(recvcounts), _size_array(rdispls),
                      _dtype_code(send[0].dtype), _stream_handle(stream))

    def bind_alltoallv_dynamic(self, send, counts, recv, row_elems, sdispls=None, rdispls=None, recvcounts=None,
                               stream=None):
        return _bound(load().hccl_alltoallv_dynamic, self.handle, _ptr_array(send), _addr(counts),
                      _addr_or_null(sdispls), _ptr_array(recv), _addr_or_null(recvcounts), _addr_or_null(rdispls),
                      row_elems, self._capacity(send, row_elems), self._capacity(recv, row_elems),
                      _dtype_code(send[0].dtype), _stream_handle(stream))

    def triggered(self, wait=None, done=None):
        """Context manager: the next work packet called inside waits for ``wait`` =
        (word, cmp, value) and writes ``done`` = (word, value) (see hccl_set_trigger)."""
        comm = self

        class _Triggered:
            def __enter__(self):
                hccl_set_trigger(comm.handle, wait, done)
                return comm

            def __exit__(self, *exc):
                hccl_set_trigger(comm.handle)   # a trigger no call consumed does not linger
                return False

        return _Triggered()

    def group(self):
        """Context manager: the collectives called inside run as one launch at its end."""
        comm = self

        class _Group:
            def __enter__(self):
                hccl_group_start(comm.handle)
                return comm

            def __exit__(self, exc_type, *exc):
                hccl_group_end(comm.handle)
                return False

        return _Group()

    def last_program(self) -> dict:
        return hccl_comm_last_program(self.handle)

    def trace(self):
        return hccl_comm_trace(self.handle)

    def program_image(self) -> bytes:
        return hccl_comm_program_image(self.handle)

    def async_error(self) -> int:
        return hccl_get_async_error(self.handle)

    def resident(self, blocks: int = 0, idle_ms: int = 0):
        """Context manager: calls inside go to a resident executor through the host doorbell
        (see hccl_resident_start); it is stopped on exit."""
        comm = self

        class _Resident:
            def __enter__(self):
                hccl_resident_start(comm.handle, blocks, idle_ms)
                return comm

            def __exit__(self, *exc):
                hccl_resident_stop(comm.handle)
                return False

        return _Resident()

    def resident_wait(self, seq: int = 0, timeout_ms: int = 0) -> None:
        hccl_resident_wait(self.handle, seq, timeout_ms)

    def resident_seq(self) -> int:
        return hccl_resident_last_seq(self.handle)
