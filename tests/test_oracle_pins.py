"""Pins for the CPU oracle: it is checked against things other than itself.

Each test ties the oracle to a library routine that implements the same definition
independently (numpy / torch IEEE conversions and float32 adds), to a closed form, to a
brute-force pure-Python loop on tiny inputs, or to an invariant of the collective
definitions (paper, Section III-B-2 "Data Path"; arithmetic of Section II-A-2 "Near Memory
Compute"). The set is chosen so that a plausible slip in the oracle -- a dropped or extra
term, a wrong block or rank index, the wrong fold order, a +0.0 seed, a bad rounding rule,
a transposed count table -- fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from workloads import alltoallv_layout, normal_bf16, normal_f32, small_int_valued, uniform_f32, zipf_counts


# ----------------------------------------------------------------------------- helpers
def _bit_patterns(lows):
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    return np.concatenate([(hi | np.uint32(lo)) for lo in lows]).view(np.float32)


def _same_bits_or_both_nan(a_bits, b_bits, as_float):
    a_nan = np.isnan(as_float(a_bits))
    b_nan = np.isnan(as_float(b_bits))
    assert np.array_equal(a_nan, b_nan)
    keep = ~a_nan
    assert np.array_equal(a_bits[keep], b_bits[keep])


def _torch_bf16_bits(x_f32):
    return torch.from_numpy(np.ascontiguousarray(x_f32, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _torch_bf16_widen(bits):
    return torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float32).numpy()


def _np_fold(rows_f32):
    """Ascending fold with numpy float32 adds (each one IEEE round-to-nearest-even)."""
    acc = rows_f32[0].copy()
    for r in range(1, rows_f32.shape[0]):
        acc = (acc + rows_f32[r]).astype(np.float32)
    return acc


# ----------------------------------------------------------------------- conversions
def test_bf16_narrowing_matches_torch_on_every_tie_class():
    # every upper half combined with remainders below, at, just above half, and extremes
    rng = np.random.default_rng(1)
    lows = [0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF] + [int(v) for v in rng.integers(0, 1 << 16, 4)]
    x = _bit_patterns(lows)
    ours = oracle.f32_to_bf16(x)
    ref = _torch_bf16_bits(x)
    _same_bits_or_both_nan(ours, ref, oracle.bf16_to_f32)


def test_bf16_widening_is_exact_for_all_encodings():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = oracle.bf16_to_f32(bits)
    ref = _torch_bf16_widen(bits)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan].view(np.uint32), ref[~nan].view(np.uint32))


def test_bf16_hand_values():
    # 1 + 2^-8 lies exactly between bf16 neighbours 1 and 1 + 2^-7: the even one (1.0) wins;
    # 1 + 3*2^-8 lies between 1 + 2^-7 and 1 + 2^-6: the even one is 1 + 2^-6.
    one = 1.0
    vals = np.array([one + 2 ** -8, one + 3 * 2 ** -8, one + 2 ** -8 + 2 ** -20, -0.0,
                     3.4028234663852886e38, np.inf], dtype=np.float32)
    got = oracle.f32_to_bf16(vals)
    assert got[0] == 0x3F80           # 1.0
    assert got[1] == 0x3F82           # 1 + 2^-6
    assert got[2] == 0x3F81           # above the tie: rounds up to 1 + 2^-7
    assert got[3] == 0x8000           # -0 keeps its sign
    assert got[4] == 0x7F80           # the largest float32 rounds past the largest bf16 to +inf
    assert got[5] == 0x7F80


def test_fp16_narrowing_matches_numpy_on_every_tie_class():
    rng = np.random.default_rng(2)
    lows = [0x0000, 0x0001, 0x0FFF, 0x1000, 0x1001, 0x2000, 0xFFFF] + [int(v) for v in rng.integers(0, 1 << 16, 4)]
    x = _bit_patterns(lows)
    ours = oracle.f32_to_f16(x)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    _same_bits_or_both_nan(ours, ref, lambda b: b.view(np.float16))


def test_fp16_narrowing_subnormal_ties():
    # values k/2 units of 2^-24: odd k are exact ties between subnormal neighbours
    k = np.arange(0, 4096, dtype=np.float64)
    x = (k * 2.0 ** -25).astype(np.float32)
    x = np.concatenate([x, -x])
    ours = oracle.f32_to_f16(x)
    ref = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(ours, ref)


def test_fp16_widening_is_exact_for_all_encodings():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = oracle.f16_to_f32(bits)
    ref = bits.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan].view(np.uint32), ref[~nan].view(np.uint32))


# ------------------------------------------------------------------- reduction order
@pytest.mark.parametrize("P", [1, 2, 3, 5, 8, 13])
def test_allreduce_fp32_is_the_ascending_numpy_fold(P):
    x = uniform_f32(P, 3001, seed=P)
    out = oracle.allreduce(x, "fp32")
    ref = _np_fold(x)
    for r in range(P):
        assert np.array_equal(out[r].view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("P", [2, 4, 8])
def test_allreduce_bf16_is_torch_widen_numpy_fold_torch_round(P):
    xb = normal_bf16(P, 4099, std=3.0, seed=10 + P)
    out = oracle.allreduce(xb, "bf16")
    wide = np.stack([_torch_bf16_widen(xb[r]) for r in range(P)])
    ref = _torch_bf16_bits(_np_fold(wide))
    for r in range(P):
        assert np.array_equal(out[r], ref)


@pytest.mark.parametrize("P", [2, 3, 8])
def test_allreduce_fp16_is_numpy_widen_fold_round(P):
    x = (normal_f32(P, 2053, std=40.0, seed=20 + P)).astype(np.float16)
    bits = x.view(np.uint16)
    out = oracle.allreduce(bits, "fp16")
    ref = _np_fold(x.astype(np.float32)).astype(np.float16).view(np.uint16)
    for r in range(P):
        assert np.array_equal(out[r], ref)


def test_fold_order_is_ascending_rank_not_any_other():
    # ranks hold 1, 1e8, -1e8. Ascending: (1 + 1e8) rounds to 1e8, then -1e8 -> 0.
    # Descending: (-1e8 + 1e8) = 0, then + 1 -> 1. Only the ascending fold gives 0.
    x = np.array([[1.0], [1e8], [-1e8]], dtype=np.float32)
    assert oracle.allreduce(x, "fp32")[0, 0] == 0.0
    y = x[::-1].copy()
    assert oracle.allreduce(y, "fp32")[0, 0] == 1.0


def test_accumulator_is_seeded_with_the_first_contributor():
    # a column of -0.0 must reduce to -0.0; a +0.0 seed would give +0.0
    for dt, bits in (("fp32", np.full((4, 3), -0.0, np.float32)),
                     ("bf16", np.full((4, 3), 0x8000, np.uint16)),
                     ("fp16", np.full((4, 3), 0x8000, np.uint16))):
        out = oracle.allreduce(bits, dt)
        if dt == "fp32":
            assert np.all(np.signbit(out))
        else:
            assert np.all(out == 0x8000)
    mixed = np.array([[-0.0], [0.0]], np.float32)
    assert not np.signbit(oracle.allreduce(mixed, "fp32")[0, 0])


@pytest.mark.parametrize("L,G", [(2, 2), (4, 2), (8, 8), (3, 5)])
def test_two_level_is_group_folds_then_partial_fold(L, G):
    P = L * G
    x = normal_f32(P, 1024, std=1.0, seed=P)
    out = oracle.allreduce(x, "fp32", group=L)
    parts = np.stack([_np_fold(x[g * L:(g + 1) * L]) for g in range(G)])
    ref = _np_fold(parts)
    assert np.array_equal(out[0].view(np.uint32), ref.view(np.uint32))
    # bf16: partials stay fp32, one rounding at the end
    xb = normal_bf16(P, 1024, seed=P + 1)
    outb = oracle.allreduce(xb, "bf16", group=L)
    wide = np.stack([_torch_bf16_widen(xb[r]) for r in range(P)])
    parts = np.stack([_np_fold(wide[g * L:(g + 1) * L]) for g in range(G)])
    assert np.array_equal(outb[0], _torch_bf16_bits(_np_fold(parts)))


def test_two_level_differs_from_flat_within_the_stated_bound():
    # both orders are recursive fp32 sums of the same P terms: each is within
    # gamma_{P-1} * sum|x| of the exact sum, and one bf16 rounding follows
    L, G = 8, 8
    P = L * G
    xb = normal_bf16(P, 20000, seed=7)
    flat = oracle.bf16_to_f32(oracle.allreduce(xb, "bf16")[0]).astype(np.float64)
    tree = oracle.bf16_to_f32(oracle.allreduce(xb, "bf16", group=L)[0]).astype(np.float64)
    wide = oracle.bf16_to_f32(xb).astype(np.float64)
    u = 2.0 ** -24
    gamma = (P - 1) * u / (1 - (P - 1) * u)
    bound = 2 * gamma * np.abs(wide).sum(axis=0)
    ulp = np.spacing(np.maximum(np.abs(flat), np.abs(tree)).astype(np.float32)).astype(np.float64) * 2 ** 16
    assert np.all(np.abs(flat - tree) <= ulp + bound)
    # in fp32 (no final rounding to hide it) the two orders really differ somewhere
    x = normal_f32(P, 20000, seed=8)
    f32_flat = oracle.allreduce(x, "fp32")[0].astype(np.float64)
    f32_tree = oracle.allreduce(x, "fp32", group=L)[0].astype(np.float64)
    assert np.any(f32_flat != f32_tree)
    assert np.all(np.abs(f32_flat - f32_tree) <= 2 * gamma * np.abs(x.astype(np.float64)).sum(axis=0))


# ----------------------------------------------------------------------- closed forms
@pytest.mark.parametrize("dt", ["fp32", "bf16", "fp16", "int32"])
@pytest.mark.parametrize("P", [1, 2, 7, 16])
def test_allreduce_of_rank_plus_one_is_triangular_number(dt, P):
    vals = np.arange(1, P + 1, dtype=np.float32)[:, None] * np.ones((1, 37), np.float32)
    if dt == "fp32":
        x = vals
    elif dt == "bf16":
        x = _torch_bf16_bits(vals)
    elif dt == "fp16":
        x = vals.astype(np.float16).view(np.uint16)
    else:
        x = vals.astype(np.int32)
    out = oracle.allreduce(x, dt)
    if dt == "bf16":
        got = oracle.bf16_to_f32(out)
    elif dt == "fp16":
        got = out.view(np.float16).astype(np.float32)
    else:
        got = out.astype(np.float64)
    assert np.all(got == P * (P + 1) // 2)


@pytest.mark.parametrize("dt", ["fp32", "bf16", "fp16"])
def test_small_integer_sums_are_exact_in_every_order(dt):
    P = 16
    v = small_int_valued(P, 5000, -8, 8, seed=3)
    exact = v.astype(np.int64).sum(axis=0)
    conv = {"fp32": (lambda a: a, lambda b: b),
            "bf16": (_torch_bf16_bits, oracle.bf16_to_f32),
            "fp16": (lambda a: a.astype(np.float16).view(np.uint16), lambda b: b.view(np.float16).astype(np.float32))}
    enc, dec = conv[dt]
    x = enc(v)
    for group in (0, 2, 4, 8):
        out = dec(oracle.allreduce(x, dt, group=group)[0])
        assert np.array_equal(out.astype(np.int64), exact)


def test_int32_sum_wraps_like_uint32_arithmetic():
    rng = np.random.default_rng(5)
    P = 9
    x = rng.integers(-2 ** 31, 2 ** 31, size=(P, 4000), dtype=np.int64).astype(np.int32)
    x[:, :4] = np.int32(2 ** 31 - 1)        # forced overflow columns
    out = oracle.allreduce(x, "int32")
    ref = x.view(np.uint32).astype(np.uint64).sum(axis=0) % (2 ** 32)
    assert np.array_equal(out[0].view(np.uint32).astype(np.uint64), ref)


def test_fp32_result_is_within_the_recursive_summation_bound_of_the_exact_sum():
    P = 8
    x = uniform_f32(P, 2000, seed=11)
    out = oracle.allreduce(x, "fp32")[0].astype(np.float64)
    exact = np.array([math.fsum(x[:, i].astype(np.float64)) for i in range(x.shape[1])])
    u = 2.0 ** -24
    gamma = (P - 1) * u / (1 - (P - 1) * u)
    assert np.all(np.abs(out - exact) <= gamma * np.abs(x.astype(np.float64)).sum(axis=0))


@pytest.mark.parametrize("op", ["max", "min"])
def test_max_min_match_numpy_without_nans(op):
    x = normal_f32(6, 999, seed=4)
    out = oracle.allreduce(x, "fp32", op=op)[0]
    ref = (np.maximum if op == "max" else np.minimum).reduce(x, axis=0)
    assert np.array_equal(out, ref)
    xi = (x * 1000).astype(np.int32)
    outi = oracle.allreduce(xi, "int32", op=op)[0]
    assert np.array_equal(outi, (np.maximum if op == "max" else np.minimum).reduce(xi, axis=0))


def test_nan_propagates():
    x = np.array([[1.0, np.nan, 2.0], [np.nan, 3.0, 4.0], [5.0, 6.0, np.nan]], np.float32)
    for op in ("sum", "max", "min"):
        assert np.all(np.isnan(oracle.allreduce(x, "fp32", op=op)[0]))


# ------------------------------------------------------------- brute force, tiny sizes
def _py_fold(vals):
    acc = np.float32(vals[0])
    for v in vals[1:]:
        acc = np.float32(acc + np.float32(v))
    return acc


@pytest.mark.parametrize("P,M", [(1, 5), (2, 1), (3, 4), (4, 7), (5, 3)])
def test_reduce_scatter_brute_force(P, M):
    x = uniform_f32(P, P * M, seed=P * 10 + M)
    out = oracle.reduce_scatter(x, "fp32")
    for c in range(P):
        for j in range(M):
            want = _py_fold([x[r][c * M + j] for r in range(P)])
            assert out[c][j].view(np.uint32) == np.float32(want).view(np.uint32)


@pytest.mark.parametrize("P,M", [(1, 3), (2, 5), (3, 1), (5, 4)])
def test_allgather_brute_force(P, M):
    x = np.arange(P * M, dtype=np.int32).reshape(P, M) * 7 + 1
    out = oracle.allgather(x)
    for r in range(P):
        for q in range(P):
            for j in range(M):
                assert out[r][q * M + j] == x[q][j]


def test_alltoallv_brute_force_with_gaps_and_zero_blocks():
    P = 4
    rng = np.random.default_rng(9)
    counts = rng.integers(0, 5, size=(P, P))
    counts[1, 2] = 0
    counts[3, 3] = 0
    lay = alltoallv_layout(counts)
    # receive layout with a gap of 3 poison elements after every block
    rdispls = np.zeros((P, P), np.int64)
    for d in range(P):
        off = 2
        for s in range(P):
            rdispls[d, s] = off
            off += lay["recvcounts"][d, s] + 3
    send = [np.arange(lay["send_len"][s], dtype=np.int32) + 1000 * (s + 1) for s in range(P)]
    recv = [np.full(int(rdispls[d].max() + lay["recvcounts"][d].max() + 8), -7, np.int32) for d in range(P)]
    expect = [r.copy() for r in recv]
    for s in range(P):
        for d in range(P):
            for i in range(counts[s, d]):
                expect[d][rdispls[d, s] + i] = send[s][lay["sdispls"][s, d] + i]
    oracle.alltoallv(send, lay["sendcounts"], lay["sdispls"], recv, lay["recvcounts"], rdispls)
    for d in range(P):
        assert np.array_equal(recv[d], expect[d])


def test_alltoallv_rejects_inconsistent_counts():
    P = 2
    counts = np.array([[1, 2], [3, 4]])
    lay = alltoallv_layout(counts)
    bad = lay["recvcounts"].copy()
    bad[0, 1] += 1
    send = [np.zeros(8, np.int32) for _ in range(P)]
    recv = [np.zeros(16, np.int32) for _ in range(P)]
    with pytest.raises(ValueError):
        oracle.alltoallv(send, lay["sendcounts"], lay["sdispls"], recv, bad, lay["rdispls"])


# ------------------------------------------------------------------------ invariants
@pytest.mark.parametrize("dt", ["fp32", "bf16"])
def test_allgather_of_reduce_scatter_equals_allreduce(dt):
    P, M = 6, 333
    x = uniform_f32(P, P * M, seed=12) if dt == "fp32" else normal_bf16(P, P * M, seed=12)
    rs = oracle.reduce_scatter(x, dt)
    ag = oracle.allgather(rs)
    ar = oracle.allreduce(x, dt)
    assert np.array_equal(ag.view(np.uint8), ar.view(np.uint8))


def test_allreduce_outputs_are_identical_on_every_rank():
    x = normal_bf16(8, 10000, seed=13)
    out = oracle.allreduce(x, "bf16")
    for r in range(1, 8):
        assert np.array_equal(out[r], out[0])


def test_p1_is_identity():
    x = normal_bf16(1, 777, seed=14)
    assert np.array_equal(oracle.allreduce(x, "bf16"), x)
    assert np.array_equal(oracle.reduce_scatter(x[:, :777], "bf16"), x)
    assert np.array_equal(oracle.allgather(x), x)


def _a2av(send, counts_sd, elems):
    P = len(send)
    lay = alltoallv_layout(counts_sd, elems)
    recv = [np.zeros(int(lay["recv_len"][d]), send[0].dtype) for d in range(P)]
    oracle.alltoallv(send, lay["sendcounts"], lay["sdispls"], recv, lay["recvcounts"], lay["rdispls"])
    return recv


def test_alltoallv_twice_with_transposed_counts_is_identity_and_conserves_bytes():
    P, R, D = 8, 3000, 16
    counts = zipf_counts(P, R, 1.1, seed=0)
    lay = alltoallv_layout(counts, D)
    send = [np.random.default_rng(s).integers(0, 2 ** 16, int(lay["send_len"][s]), dtype=np.uint16) for s in range(P)]
    recv = _a2av(send, counts, D)
    assert sum(r.nbytes for r in recv) == sum(s.nbytes for s in send)
    # multiset of rows is preserved
    rows_in = np.sort(np.concatenate([s.reshape(-1, D) for s in send]).view(np.dtype((np.void, 2 * D))).ravel())
    rows_out = np.sort(np.concatenate([r.reshape(-1, D) for r in recv]).view(np.dtype((np.void, 2 * D))).ravel())
    assert np.array_equal(rows_in, rows_out)
    back = _a2av(recv, counts.T.copy(), D)
    for s in range(P):
        assert np.array_equal(back[s], send[s])


def test_alltoallv_with_uniform_counts_is_a_block_transpose():
    P, B = 5, 6
    x = np.arange(P * P * B, dtype=np.int32).reshape(P, P * B)
    recv = _a2av([x[s].copy() for s in range(P)], np.full((P, P), B), 1)
    ref = torch.from_numpy(x.reshape(P, P, B)).transpose(0, 1).contiguous().reshape(P, P * B).numpy()
    assert np.array_equal(np.stack(recv), ref)


def test_reduce_scatter_rejects_bad_group():
    x = uniform_f32(6, 12, seed=1)
    with pytest.raises(ValueError):
        oracle.allreduce(x, "fp32", group=4)   # 6 ranks do not split into groups of 4
