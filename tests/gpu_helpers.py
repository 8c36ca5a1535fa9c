"""Helpers for the GPU parity tests: move seeded host arrays to the device and back.

Element data travels as raw bits (uint16 for bf16 / fp16), so nothing here rounds or
converts values: what the oracle sees and what the GPU sees are the same bits.
"""
import numpy as np
import torch

TORCH_DTYPE = {"bf16": torch.bfloat16, "fp16": torch.float16, "fp32": torch.float32, "int32": torch.int32}
NP_BITS = {"bf16": np.uint16, "fp16": np.uint16, "fp32": np.float32, "int32": np.int32}
GUARD = 64  # poison elements before and after every output buffer


def to_device(bits: np.ndarray, dt: str, device="cuda:0") -> torch.Tensor:
    """1-D host bits -> device tensor of the element type (bit-identical)."""
    bits = np.ascontiguousarray(bits)
    if dt in ("bf16", "fp16"):
        t = torch.from_numpy(bits.view(np.int16).copy()).to(device)
        return t.view(TORCH_DTYPE[dt])
    return torch.from_numpy(bits.copy()).to(device)


def to_host(t: torch.Tensor, dt: str) -> np.ndarray:
    t = t.detach().contiguous()
    if dt in ("bf16", "fp16"):
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


class Guarded:
    """A device buffer of n elements with GUARD poison elements on both sides."""

    POISON = {"bf16": 0x7FA5, "fp16": 0x7DA5, "fp32": np.float32(np.nan), "int32": np.int32(-0x5A5A5A5B)}

    def __init__(self, n: int, dt: str, device="cuda:0", fill=None):
        self.n, self.dt = n, dt
        host = np.empty(n + 2 * GUARD, dtype=NP_BITS[dt])
        if dt == "fp32":
            host.view(np.uint32)[:] = 0x7FA5A5A5
        else:
            host[:] = self.POISON[dt]
        if fill is not None:
            host[GUARD:GUARD + n] = fill
        self.host_init = host.copy()
        self.full = to_device(host, dt, device)
        self.view = self.full[GUARD:GUARD + n]

    def result(self) -> np.ndarray:
        return to_host(self.view, self.dt)

    def guards_intact(self) -> bool:
        h = to_host(self.full, self.dt)
        a = h[:GUARD].view(np.uint8) if h.dtype != np.uint8 else h[:GUARD]
        b = self.host_init[:GUARD].view(np.uint8)
        c = h[GUARD + self.n:].view(np.uint8)
        d = self.host_init[GUARD + self.n:].view(np.uint8)
        return np.array_equal(a, b) and np.array_equal(c, d)


def same_bits(a: np.ndarray, b: np.ndarray, dt: str, nan_equal=True) -> bool:
    """Bitwise equality; with nan_equal, any NaN matches any NaN (payloads are not compared)."""
    if a.shape != b.shape:
        return False
    if dt == "int32":
        return np.array_equal(a, b)
    ua = a.view(np.uint16 if dt in ("bf16", "fp16") else np.uint32)
    ub = b.view(np.uint16 if dt in ("bf16", "fp16") else np.uint32)
    if not nan_equal:
        return np.array_equal(ua, ub)
    if dt == "fp32":
        na, nb = np.isnan(a), np.isnan(b)
    elif dt == "bf16":
        na = ((ua & 0x7F80) == 0x7F80) & ((ua & 0x7F) != 0)
        nb = ((ub & 0x7F80) == 0x7F80) & ((ub & 0x7F) != 0)
    else:
        na = ((ua & 0x7C00) == 0x7C00) & ((ua & 0x3FF) != 0)
        nb = ((ub & 0x7C00) == 0x7C00) & ((ub & 0x3FF) != 0)
    if not np.array_equal(na, nb):
        return False
    return np.array_equal(ua[~na], ub[~nb])


def first_mismatch(a: np.ndarray, b: np.ndarray) -> str:
    idx = np.nonzero(a.view(np.uint16 if a.itemsize == 2 else np.uint32) != b.view(np.uint16 if b.itemsize == 2 else np.uint32))[0]
    if idx.size == 0:
        return "no mismatch"
    i = int(idx[0])
    return f"{idx.size} mismatches, first at {i}: got {a[i]!r} want {b[i]!r}"


class MaskedStream:
    """A HIP stream confined to the first `per_xcd` CUs of every XCD (mask bit i selects a CU of
    XCD i mod 8), at the default priority; destroyed on exit."""

    def __init__(self, per_xcd=2):
        import ctypes

        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipExtStreamCreateWithCUMask.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32,
                                                           ctypes.POINTER(ctypes.c_uint32)]
        self._hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
        ncu = torch.cuda.get_device_properties(0).multi_processor_count
        words = (ncu + 31) // 32
        bits = [0] * words
        for i in range(8 * per_xcd):
            bits[i // 32] |= 1 << (i % 32)
        arr = (ctypes.c_uint32 * words)(*bits)
        handle = ctypes.c_void_p()
        rc = self._hip.hipExtStreamCreateWithCUMask(ctypes.byref(handle), words, arr)
        if rc != 0:
            raise RuntimeError(f"hipExtStreamCreateWithCUMask failed ({rc})")
        self.handle = handle.value
        self.stream = torch.cuda.ExternalStream(self.handle)

    def __enter__(self):
        return self.stream

    def __exit__(self, *exc):
        self.stream.synchronize()
        self._hip.hipStreamDestroy(self.handle)
        return False


class SideStream:
    """A non-blocking HIP stream at the default priority (work on it never waits for the null
    stream, and the null stream never waits for it); destroyed on exit."""

    def __init__(self):
        import ctypes

        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipStreamCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32]
        self._hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
        handle = ctypes.c_void_p()
        rc = self._hip.hipStreamCreateWithFlags(ctypes.byref(handle), 1)  # hipStreamNonBlocking
        if rc != 0:
            raise RuntimeError(f"hipStreamCreateWithFlags failed ({rc})")
        self.handle = handle.value
        self.stream = torch.cuda.ExternalStream(self.handle)

    def __enter__(self):
        return self.stream

    def __exit__(self, *exc):
        self.stream.synchronize()
        self._hip.hipStreamDestroy(self.handle)
        return False
