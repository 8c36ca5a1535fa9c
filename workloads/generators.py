"""Seeded input generators (numpy PCG64). No collective arithmetic lives here.

Recipe, shared by every consumer (host generators, used up to tens of millions of values):
  * one ``numpy.random.SeedSequence(seed)`` is spawned into P child sequences; rank r draws
    its values from ``Generator(PCG64(child[r]))``, so ranks can be generated in parallel and
    a rank's data does not depend on P's other ranks being drawn;
  * bf16 / fp16 values are drawn as float32 and rounded to nearest-even by torch's CPU
    conversion (element bits are returned as uint16);
  * uniform [-1, 1) float32 values are ``random(float32) * 2 - 1``: random() yields k * 2^-24,
    so the affine map is exact and never reaches 1.0.

Device generators (full-size workloads of hundreds of millions of values, where host
generation would take minutes): rank r draws from ``torch.Generator(device)`` seeded with
``seed * 1_000_003 + r`` (torch's Philox counter-based generator), in float32, then rounds to
bf16 with torch. Callers that need the values on the host copy the device tensor back; the
values are the same bits on both sides.
"""
from __future__ import annotations

import concurrent.futures as _cf
import os

import numpy as np

_MAX_THREADS = max(1, min(16, os.cpu_count() or 1))


def _rank_generators(P: int, seed: int):
    children = np.random.SeedSequence(seed).spawn(P)
    return [np.random.Generator(np.random.PCG64(c)) for c in children]


def _fill_rows(P: int, N: int, out_dtype, fill):
    out = np.empty((P, N), dtype=out_dtype)
    if P == 0 or N == 0:
        return out
    with _cf.ThreadPoolExecutor(max_workers=min(P, _MAX_THREADS)) as ex:
        list(ex.map(lambda r: fill(r, out[r]), range(P)))
    return out


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest-even, torch CPU) and return the bits."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def uniform_f32(P: int, N: int, seed: int = 0) -> np.ndarray:
    """(P, N) float32, uniform in [-1, 1)."""
    gens = _rank_generators(P, seed)

    def fill(r, row):
        gens[r].random(out=row, dtype=np.float32)
        row *= np.float32(2.0)
        row -= np.float32(1.0)

    return _fill_rows(P, N, np.float32, fill)


def normal_f32(P: int, N: int, mean: float = 0.0, std: float = 1.0, seed: int = 0) -> np.ndarray:
    """(P, N) float32 draws of N(mean, std)."""
    gens = _rank_generators(P, seed)

    def fill(r, row):
        gens[r].standard_normal(out=row, dtype=np.float32)
        if std != 1.0:
            row *= np.float32(std)
        if mean != 0.0:
            row += np.float32(mean)

    return _fill_rows(P, N, np.float32, fill)


def normal_bf16(P: int, N: int, mean: float = 0.0, std: float = 1.0, seed: int = 0) -> np.ndarray:
    """(P, N) bfloat16 bits (uint16) of N(mean, std) draws rounded to nearest-even."""
    gens = _rank_generators(P, seed)

    def fill(r, row):
        tmp = gens[r].standard_normal(N, dtype=np.float32)
        if std != 1.0:
            tmp *= np.float32(std)
        if mean != 0.0:
            tmp += np.float32(mean)
        row[:] = bf16_bits_from_f32(tmp)

    return _fill_rows(P, N, np.uint16, fill)


def small_int_valued(P: int, N: int, lo: int = -8, hi: int = 8, seed: int = 0) -> np.ndarray:
    """(P, N) float32 holding small integers in [lo, hi): every sum of them is exact in
    bf16 / fp16 / fp32 as long as the running magnitude stays below 256."""
    gens = _rank_generators(P, seed)

    def fill(r, row):
        row[:] = gens[r].integers(lo, hi, size=N).astype(np.float32)

    return _fill_rows(P, N, np.float32, fill)


def row_ids_int32(P: int, rows: int, seed: int = 0) -> np.ndarray:
    """(P, rows) int32 row ids, uniform in [0, 2^31)."""
    gens = _rank_generators(P, seed)

    def fill(r, row):
        row[:] = gens[r].integers(0, 2**31, size=rows, dtype=np.int64).astype(np.int32)

    return _fill_rows(P, rows, np.int32, fill)


def zipf_counts(P: int, rows_per_rank: int, s: float = 1.1, seed: int = 0) -> np.ndarray:
    """(P, P) int64 row counts, indexed [src, dst].

    Every source sends exactly ``rows_per_rank`` rows. Each row of source ``src`` picks a
    popularity rank k in 1..P with probability proportional to k^-s (a finite Zipf law), and
    rank k is mapped to a destination by a per-source random permutation; the counts are the
    resulting multinomial draw. Zero counts are allowed.
    """
    gens = _rank_generators(P, seed)
    k = np.arange(1, P + 1, dtype=np.float64)
    p = k ** (-float(s))
    p /= p.sum()
    counts = np.zeros((P, P), dtype=np.int64)
    for src in range(P):
        g = gens[src]
        perm = g.permutation(P)
        draw = g.multinomial(rows_per_rank, p)
        counts[src, perm] = draw
    return counts


def alltoallv_layout(row_counts: np.ndarray, elems_per_row: int = 1) -> dict:
    """Element counts / displacements for an AllToAllv whose send buffers are laid out
    destination-major and whose receive buffers are laid out source-major.

    Returns (P, P) int64 arrays: ``sendcounts[s, d]``, ``sdispls[s, d]`` (send side, indexed
    [src, dst]) and ``recvcounts[d, s]``, ``rdispls[d, s]`` (receive side, indexed [dst, src]),
    plus the per-rank send and receive lengths in elements.
    """
    c = np.asarray(row_counts, dtype=np.int64) * int(elems_per_row)
    P = c.shape[0]
    sendcounts = c.copy()
    sdispls = np.zeros_like(c)
    sdispls[:, 1:] = np.cumsum(c, axis=1)[:, :-1]
    recvcounts = c.T.copy()
    rdispls = np.zeros_like(c)
    rdispls[:, 1:] = np.cumsum(recvcounts, axis=1)[:, :-1]
    return {
        "sendcounts": sendcounts,
        "sdispls": sdispls,
        "recvcounts": recvcounts,
        "rdispls": rdispls,
        "send_len": c.sum(axis=1),
        "recv_len": c.sum(axis=0),
        "P": P,
    }


def device_rank_seed(seed: int, r: int) -> int:
    return seed * 1_000_003 + r


def device_normal_bf16(P: int, N: int, mean: float = 0.0, std: float = 1.0, seed: int = 0,
                       device: str = "cuda:0"):
    """List of P device tensors (bfloat16, N elements) of N(mean, std) draws."""
    import torch

    out = []
    for r in range(P):
        g = torch.Generator(device=device)
        g.manual_seed(device_rank_seed(seed, r))
        x = torch.randn(N, generator=g, device=device, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        if mean != 0.0:
            x.add_(mean)
        out.append(x.to(torch.bfloat16))
        del x
    return out


def device_uniform_f32(P: int, N: int, seed: int = 0, device: str = "cuda:0"):
    """List of P device tensors (float32, N elements), uniform in [-1, 1)."""
    import torch

    out = []
    for r in range(P):
        g = torch.Generator(device=device)
        g.manual_seed(device_rank_seed(seed, r))
        x = torch.rand(N, generator=g, device=device, dtype=torch.float32)
        out.append(x.mul_(2.0).sub_(1.0))
    return out
