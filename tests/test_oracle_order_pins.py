"""Pins for the oracle's other fold orders: ring (rotated per shard), recursive-halving tree,
and per-combine re-quantisation to the buffer type (paper, Section III-B-2 ring AllReduce;
Section II-A-2 NMC re-quantisation). Each order is checked against an independent numpy /
torch formulation, closed forms and hand-built cancellation cases that tell the orders apart.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import normal_bf16, normal_f32, small_int_valued


def _f32_fold(rows):
    acc = rows[0].copy()
    for r in range(1, rows.shape[0]):
        acc = (acc + rows[r]).astype(np.float32)
    return acc


def _bf16_round(x):
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


def _widen(bits):
    return torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float32).numpy()


def _to_bits(x):
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _halving(rows, rnd=lambda v: v):
    v = [rows[r].copy() for r in range(rows.shape[0])]
    d = len(v) // 2
    while d >= 1:
        for r in range(d):
            v[r] = rnd((v[r] + v[r + d]).astype(np.float32))
        d //= 2
    return v[0]


@pytest.mark.parametrize("P", [1, 2, 3, 5, 8])
def test_ring_order_reduce_scatter_is_the_rotated_numpy_fold(P):
    M = 777
    x = normal_f32(P, P * M, seed=50 + P)
    out = oracle.reduce_scatter_ordered(x, "fp32", order="ring")
    for c in range(P):
        block = x[:, c * M:(c + 1) * M]
        rot = np.roll(block, -((c + 1) % P), axis=0)      # rows c+1, c+2, ..., c
        want = _f32_fold(rot)
        assert np.array_equal(out[c].view(np.uint32), want.view(np.uint32))


def test_ring_order_allreduce_rotates_per_shard():
    P, N, q = 4, 1000, 256
    x = normal_f32(P, N, seed=60)
    out = oracle.allreduce_ordered(x, "fp32", order="ring", shard=q)
    for i0 in range(0, N, q):
        c = i0 // q
        rot = np.roll(x[:, i0:i0 + q], -((c + 1) % P), axis=0)
        assert np.array_equal(out[0, i0:i0 + q].view(np.uint32), _f32_fold(rot).view(np.uint32))


@pytest.mark.parametrize("P", [1, 2, 4, 8, 16, 64])
def test_halving_order_is_the_distance_halving_tree(P):
    x = normal_f32(P, 3001, seed=70 + P)
    out = oracle.allreduce_ordered(x, "fp32", order="halving")
    assert np.array_equal(out[0].view(np.uint32), _halving(x).view(np.uint32))


def test_orders_are_told_apart_by_cancellation():
    # ring (shard 0 of a 3-rank reduce-scatter) starts at rank 1: (1e8 + -1e8) + 1 = 1;
    # ascending gives (1 + 1e8) + -1e8 = 0
    x = np.array([[1.0, 0, 0], [1e8, 0, 0], [-1e8, 0, 0]], np.float32)   # block 0 = column 0
    assert oracle.reduce_scatter_ordered(x, "fp32", order="ring")[0, 0] == 1.0
    assert oracle.reduce_scatter_ordered(x, "fp32")[0, 0] == 0.0
    # halving on [1e8, 1, -1e8, 1]: (1e8 + -1e8) + (1 + 1) = 2; the distance-doubling tree
    # (1e8 + 1) + (-1e8 + 1) = 0; ascending ((1e8 + 1) - 1e8) + 1 = 1
    y = np.array([[1e8], [1.0], [-1e8], [1.0]], np.float32)
    assert oracle.allreduce_ordered(y, "fp32", order="halving")[0, 0] == 2.0
    assert oracle.allreduce(y, "fp32")[0, 0] == 1.0


@pytest.mark.parametrize("order", ["ascending", "ring", "halving"])
def test_requant_rounds_every_partial_to_bf16(order):
    P = 8
    xb = normal_bf16(P, 4096, std=3.0, seed=80)
    wide = np.stack([_widen(xb[r]) for r in range(P)])
    out = oracle.allreduce_ordered(xb, "bf16", order=order, shard=4096, requant=True)
    if order == "ascending":
        acc = wide[0].copy()
        for r in range(1, P):
            acc = _bf16_round((acc + wide[r]).astype(np.float32))
        want = acc
    elif order == "ring":
        rot = np.roll(wide, -1, axis=0)                      # one shard: c = 0, start at rank 1
        acc = rot[0].copy()
        for r in range(1, P):
            acc = _bf16_round((acc + rot[r]).astype(np.float32))
        want = acc
    else:
        want = _halving(wide, _bf16_round)
    assert np.array_equal(out[0], _to_bits(want))
    # and it really differs from rounding only once
    once = oracle.allreduce_ordered(xb, "bf16", order=order, shard=4096)
    assert not np.array_equal(out[0], once[0])


def _group_partials(wide, group, rnd):
    """Each run of `group` consecutive ranks folded ascending, `rnd` applied after every add."""
    parts = []
    for g0 in range(0, wide.shape[0], group):
        acc = wide[g0].copy()
        for r in range(g0 + 1, g0 + group):
            acc = rnd((acc + wide[r]).astype(np.float32))
        parts.append(acc)
    return parts


@pytest.mark.parametrize("group", [2, 4])
def test_two_level_requant_rounds_inside_and_across_groups(group):
    """Two-level order with re-quantisation (every NMC result rounded to the buffer type): the
    group partials are rounded after every in-group add, and so is every add of the
    cross-group fold. Each of the two roundings is shown to matter on its own."""
    P = 8
    xb = normal_bf16(P, 8192, std=3.0, seed=81 + group)
    wide = np.stack([_widen(xb[r]) for r in range(P)])
    out = oracle.allreduce_ordered(xb, "bf16", order="two_level", group=group, requant=True)
    parts = _group_partials(wide, group, _bf16_round)
    tot = parts[0]
    for p in parts[1:]:
        tot = _bf16_round((tot + p).astype(np.float32))
    assert np.array_equal(out[0], _to_bits(tot))
    # in-group rounding only: the cross-group fold in FP32, rounded once at the end
    cross_f32 = parts[0]
    for p in parts[1:]:
        cross_f32 = (cross_f32 + p).astype(np.float32)
    if len(parts) > 2:   # with two groups the one cross-group add is rounded either way
        assert not np.array_equal(out[0], _to_bits(cross_f32))
    # cross-group rounding only: FP32 group partials
    raw = _group_partials(wide, group, lambda v: v)
    tot_raw = raw[0]
    for p in raw[1:]:
        tot_raw = _bf16_round((tot_raw + p).astype(np.float32))
    assert not np.array_equal(out[0], _to_bits(tot_raw))
    # and the two-level order without re-quantisation differs too
    assert not np.array_equal(out[0], oracle.allreduce_ordered(xb, "bf16", order="two_level", group=group)[0])


def test_requant_is_a_no_op_for_fp32_and_int32():
    x = normal_f32(8, 999, seed=90)
    a = oracle.allreduce_ordered(x, "fp32", order="ring", shard=100, requant=True)
    b = oracle.allreduce_ordered(x, "fp32", order="ring", shard=100)
    assert np.array_equal(a, b)
    xi = (x * 1000).astype(np.int32)
    assert np.array_equal(oracle.allreduce_ordered(xi, "int32", order="halving", requant=True),
                          oracle.allreduce_ordered(xi, "int32", order="halving"))


@pytest.mark.parametrize("order", ["ring", "halving", "two_level"])
def test_small_integer_sums_are_exact_in_every_order_with_or_without_requant(order):
    P = 8
    v = small_int_valued(P, 3000, -4, 4, seed=91)
    bits = _to_bits(v)
    exact = v.astype(np.int64).sum(axis=0)
    for requant in (False, True):
        out = oracle.allreduce_ordered(bits, "bf16", order=order, group=4, shard=1000, requant=requant)
        assert np.array_equal(_widen(out[0]).astype(np.int64), exact)


def test_ordered_entry_points_match_the_plain_ones_for_ascending_and_two_level():
    x = normal_bf16(8, 5000, seed=92)
    assert np.array_equal(oracle.allreduce_ordered(x, "bf16"), oracle.allreduce(x, "bf16"))
    assert np.array_equal(oracle.allreduce_ordered(x, "bf16", order="two_level", group=4),
                          oracle.allreduce(x, "bf16", group=4))
    y = normal_bf16(4, 4 * 300, seed=93)
    assert np.array_equal(oracle.reduce_scatter_ordered(y, "bf16"), oracle.reduce_scatter(y, "bf16"))


def test_halving_rejects_non_power_of_two_ranks():
    with pytest.raises(ValueError):
        oracle.allreduce_ordered(normal_f32(6, 10, seed=1), "fp32", order="halving")
