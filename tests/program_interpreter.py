"""A CPU interpreter of compiled descriptor programs (test infrastructure).

It decodes the packed image the library uploads (hccl_comm_program_image) and runs its tiles on
host buffers in an order drawn at random among those the program's dependencies allow: a tile
starts only when every tile it waits for has finished (DEP_TILE: the tile with the same index
of the named step; DEP_ALL: every tile of it) and every tile of the earlier phases (launches)
has finished. So it checks what the compiler promises, that
the program computes the collective under any schedule the executor may produce, with the
arithmetic written out here once more from the step semantics:

* COPY: the bytes of the source range go to every destination.
* REDUCE: per element, the sources are widened to FP32 (INT32 stays integer) and combined in
  list order (``group`` = L: each run of L folded into a partial, then the partials; FOLD_PAIRWISE:
  a complete binary tree over the list), every combination rounded to the destination type
  when ``requant`` is set; the result is rounded once (nearest, ties to even) to the
  destination type and stored to every destination.

It shares nothing with the oracle or the HIP library (its own conversions, its own folds), and
it does not run AllToAllvDynamic steps.
"""
from __future__ import annotations

import numpy as np

OP_COPY, OP_REDUCE, OP_DYN_COPY = 0, 1, 4
DT_BF16, DT_FP16, DT_FP32, DT_INT32 = 0, 1, 2, 3
RO_SUM, RO_MAX, RO_MIN = 0, 1, 2
FOLD_LIST, FOLD_PAIRWISE = 0, 1
DEP_ALL, DEP_TILE = 0, 1
ES = {DT_BF16: 2, DT_FP16: 2, DT_FP32: 4, DT_INT32: 4}

HEADER = np.dtype([("magic", "<u4"), ("version", "<u4"), ("ndesc", "<u4"), ("ntiles", "<u4"), ("noperand", "<u4"),
                   ("ndep", "<u4"), ("flags", "<u4"), ("nstate", "<u4"), ("off_desc", "<u8"), ("off_operand", "<u8"),
                   ("off_dep", "<u8"), ("off_tile_desc", "<u8"), ("total_bytes", "<u8"), ("scratch_bytes", "<u8"),
                   ("off_aux", "<u8"), ("naux", "<u4"), ("nphase", "<u4"), ("off_phase", "<u8"), ("pad", "<u8")])
DESC = np.dtype([("op", "u1"), ("redop", "u1"), ("flags", "u1"), ("sig", "u1"), ("nsrc", "<u2"), ("ndst", "<u2"),
                 ("group", "<u2"), ("ndep", "<u2"), ("src", "<u4"), ("dst", "<u4"), ("dep", "<u4"), ("tile0", "<u4"),
                 ("ntiles", "<u4"), ("tile_elems", "<u4"), ("pad0", "<u4"), ("nelem", "<u8"), ("fold", "<u4"),
                 ("requant", "<u4"), ("aux", "<u4"), ("pad1", "<u4")])
OPERAND = np.dtype([("buf", "<u4"), ("dtype", "<u4"), ("offset", "<u8")])
DEP = np.dtype([("desc", "<u4"), ("kind", "<u4"), ("expected", "<u4"), ("state", "<u4")])
assert HEADER.itemsize == 112 and DESC.itemsize == 64 and OPERAND.itemsize == 16 and DEP.itemsize == 16


class Program:
    def phase_of(self, tile: int) -> int:
        return int(np.searchsorted(self.phase_tile, tile, side="right")) - 1

    def __init__(self, image: bytes):
        raw = np.frombuffer(image, dtype=np.uint8).copy()
        self.h = np.frombuffer(image, dtype=HEADER, count=1)[0]
        assert int(self.h["magic"]) == 0x4C434348 and int(self.h["total_bytes"]) == len(image)
        nd, no, ndep = int(self.h["ndesc"]), int(self.h["noperand"]), int(self.h["ndep"])
        self.descs = raw[int(self.h["off_desc"]):][: nd * 64].view(DESC)
        self.ops = raw[int(self.h["off_operand"]):][: no * 16].view(OPERAND)
        self.deps = raw[int(self.h["off_dep"]):][: ndep * 16].view(DEP)
        self.tile_desc = raw[int(self.h["off_tile_desc"]):][: int(self.h["ntiles"]) * 4].view("<u4")
        self.scratch_bytes = int(self.h["scratch_bytes"])
        nph = int(self.h["nphase"])
        # phase q runs tiles [phase_tile[q], phase_tile[q + 1])
        self.phase_tile = raw[int(self.h["off_phase"]):][: (nph + 1) * 4].view("<u4").astype(np.int64)
        assert nph >= 1 and self.phase_tile[0] == 0 and self.phase_tile[-1] == int(self.h["ntiles"])
        assert (np.diff(self.phase_tile) >= 0).all()


# ------------------------------------------------------------------------ element types
def _widen(raw: np.ndarray, dt: int) -> np.ndarray:
    if dt == DT_BF16:
        return (raw.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    if dt == DT_FP16:
        return raw.view(np.float16).astype(np.float32)
    if dt == DT_FP32:
        return raw.view(np.float32).copy()
    return raw.view(np.int32).copy()


def _narrow(v: np.ndarray, dt: int) -> np.ndarray:
    """Values in the accumulation type -> raw elements of type dt (round to nearest even)."""
    if dt == DT_BF16:
        u = v.astype(np.float32).view(np.uint32)
        nan = (u & 0x7FFFFFFF) > 0x7F800000
        rounded = ((u.astype(np.uint64) + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
        quiet = ((u >> 16) | 0x40).astype(np.uint16)
        return np.where(nan, quiet, rounded)
    if dt == DT_FP16:
        with np.errstate(over="ignore"):
            return v.astype(np.float32).astype(np.float16).view(np.uint16)
    if dt == DT_FP32:
        return v.astype(np.float32)
    return v.astype(np.int32)


def _combine(op: int, a: np.ndarray, x: np.ndarray) -> np.ndarray:
    if a.dtype == np.int32:
        if op == RO_SUM:
            return (a.view(np.uint32) + x.view(np.uint32)).view(np.int32)
        return np.maximum(a, x) if op == RO_MAX else np.minimum(a, x)
    if op == RO_SUM:
        return (a + x).astype(np.float32)
    better = (x > a) if op == RO_MAX else (x < a)
    return np.where(np.isnan(a), a, np.where(np.isnan(x), x, np.where(better, x, a))).astype(np.float32)


# --------------------------------------------------------------------------- execution
class Interpreter:
    def __init__(self, prog: Program, buffers: dict):
        """buffers: buffer id -> writable uint8 numpy array (the scratch id included)."""
        self.p = prog
        self.b = buffers

    def _view(self, op, first: int, n: int) -> np.ndarray:
        es = ES[int(op["dtype"])]
        lo = int(op["offset"]) + first * es
        return self.b[int(op["buf"])][lo: lo + n * es]

    def run_tile(self, t: int):
        d = int(self.p.tile_desc[t])
        D = self.p.descs[d]
        k = t - int(D["tile0"])
        te, nelem = int(D["tile_elems"]), int(D["nelem"])
        first = k * te
        n = min(te, nelem - first)
        if n <= 0:
            return
        srcs = self.p.ops[int(D["src"]): int(D["src"]) + int(D["nsrc"])]
        dsts = self.p.ops[int(D["dst"]): int(D["dst"]) + int(D["ndst"])]
        op = int(D["op"])
        if op == OP_COPY:
            data = self._view(srcs[0], first, n).copy()
            for o in dsts:
                self._view(o, first, n)[:] = data
            return
        assert op == OP_REDUCE, f"step kind {op} is not interpreted"
        to = int(dsts[0]["dtype"])
        req = bool(D["requant"]) and to in (DT_BF16, DT_FP16)
        redop = int(D["redop"])

        def combq(a, x):
            v = _combine(redop, a, x)
            return _widen(_narrow(v, to).view(np.uint8), to) if req else v

        vals = [_widen(self._view(o, first, n), int(o["dtype"])) for o in srcs]
        if int(D["fold"]) == FOLD_PAIRWISE:
            level = vals
            while len(level) > 1:
                level = [combq(level[i], level[i + 1]) for i in range(0, len(level), 2)]
            tot = level[0]
        else:
            L = int(D["group"]) or len(vals)
            tot = None
            for g0 in range(0, len(vals), L):
                part = vals[g0]
                for x in vals[g0 + 1: g0 + L]:
                    part = combq(part, x)
                tot = part if tot is None else combq(tot, part)
        out = _narrow(tot, to).view(np.uint8)
        for o in dsts:
            self._view(o, first, n)[:] = out

    def run(self, rng: np.random.Generator):
        """Every tile once, phase after phase, in a random order the dependencies allow."""
        p = self.p
        ntiles = len(p.tile_desc)
        nd = len(p.descs)
        done_tiles = np.zeros(ntiles, bool)
        done_count = np.zeros(nd, np.int64)
        # what each tile waits for, and who waits for what
        waits = [[] for _ in range(ntiles)]
        waiters_tile = [[] for _ in range(ntiles)]
        waiters_desc = [[] for _ in range(nd)]
        for t in range(ntiles):
            d = int(p.tile_desc[t])
            D = p.descs[d]
            k = t - int(D["tile0"])
            for e in p.deps[int(D["dep"]): int(D["dep"]) + int(D["ndep"])]:
                src = int(e["desc"])
                assert src < d, "a step waits for a later step"
                assert p.phase_of(int(p.descs[src]["tile0"])) == p.phase_of(t), "a wait across phases"
                if int(e["kind"]) == DEP_TILE:
                    st = int(p.descs[src]["tile0"]) + k
                    assert k < int(p.descs[src]["ntiles"]), "per-tile wait on a missing tile"
                    waits[t].append(("t", st))
                    waiters_tile[st].append(t)
                else:
                    waits[t].append(("d", src))
                    waiters_desc[src].append(t)
        missing = np.array([len(w) for w in waits])
        order = []
        for q in range(len(p.phase_tile) - 1):
            lo, hi = int(p.phase_tile[q]), int(p.phase_tile[q + 1])
            ready = [t for t in range(lo, hi) if missing[t] == 0]
            while ready:
                i = int(rng.integers(len(ready)))
                ready[i], ready[-1] = ready[-1], ready[i]
                t = ready.pop()
                self.run_tile(t)
                order.append(t)
                done_tiles[t] = True
                d = int(p.tile_desc[t])
                done_count[d] += 1
                woken = list(waiters_tile[t])
                if done_count[d] == int(p.descs[d]["ntiles"]):
                    woken += waiters_desc[d]
                for w in woken:
                    missing[w] -= 1
                    if missing[w] == 0:
                        ready.append(w)
            assert done_tiles[lo:hi].all(), "some tiles never became ready (a dependency cycle or a missing producer)"
        assert done_tiles.all()
        return order
