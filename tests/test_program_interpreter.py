"""Compiled programs run by a CPU interpreter, in random orders their dependencies allow.

The programs come from host-only communicators (no GPU): the packed image the library would
upload is decoded and executed tile by tile on host buffers (tests/program_interpreter.py),
three times per program with different random schedules, and the outputs must equal the
oracle's bit for bit. This checks the lowering and fusion passes value by value under every
interleaving the executor may produce; the validator checks the same programs structurally.
"""
import numpy as np
import pytest

import oracle
import paper_2608_00358_amd as H
from program_interpreter import Interpreter, Program
from workloads import alltoallv_layout, normal_bf16, normal_f32, small_int_valued, zipf_counts

ES = {"bf16": 2, "fp16": 2, "fp32": 4, "int32": 4}
STORE = {"bf16": np.uint16, "fp16": np.uint16, "fp32": np.float32, "int32": np.int32}
SMALL = dict(chunk_bytes=1024, tile_bytes=1024)
SEEDS = (1, 2, 3)


def fake(P, base):
    return [base + i * (1 << 36) for i in range(P)]


def inputs(P, n, dt, seed):
    if dt == "bf16":
        return normal_bf16(P, n, std=2.0, seed=seed)
    if dt == "fp16":
        return np.ascontiguousarray(normal_f32(P, n, seed=seed).astype(np.float16)).view(np.uint16)
    if dt == "fp32":
        return normal_f32(P, n, seed=seed)
    return small_int_valued(P, n, -2 ** 20, 2 ** 20, seed=seed).astype(np.int32)


def shard(n, P):
    q = -(-n // P)
    return -(-q // 64) * 64


def run_program(image, send, recv_sizes, seed, group_layout=None):
    """send: list (per buffer id 0..P-1) of host arrays; recv buffers start zeroed.
    group_layout: list of (P, send arrays, receive sizes) per call of a group."""
    prog = Program(image)
    bufs = {}
    calls = group_layout or [(len(send), send, recv_sizes)]
    base = 0
    outs = []
    for P, snd, rsz in calls:
        for r in range(P):
            bufs[base + r] = np.ascontiguousarray(snd[r]).view(np.uint8).copy()
            bufs[base + P + r] = np.zeros(rsz[r], np.uint8)
        outs.append([base + P + r for r in range(P)])
        base += 2 * P
    bufs[base] = np.full(max(1, prog.scratch_bytes), 0xA5, np.uint8)   # scratch: garbage at start
    Interpreter(prog, bufs).run(np.random.default_rng(seed))
    return [[bufs[i] for i in ids] for ids in outs]


def check(got_bytes, want, dt):
    for r, (g, w) in enumerate(zip(got_bytes, want)):
        w = np.ascontiguousarray(w, dtype=STORE[dt])
        assert np.array_equal(g.view(np.uint8), w.view(np.uint8)), f"rank {r} differs from the oracle"


ALLREDUCE = [
    ("ring", dict(algo="ring", fuse=0), "ascending"),
    ("ring one launch", dict(algo="ring", fuse=0, phases="one"), "ascending"),
    ("two-level one launch", dict(algo="two_level", group_size=4, fuse=0, phases="one"), "two_level"),
    ("rhd butterfly one launch", dict(algo="rhd", order="halving", fuse=0, phases="one"), "halving"),
    ("two-level fused, copies split", dict(algo="two_level", group_size=2, phases="levels"), "two_level"),
    ("ring fused", dict(algo="ring"), "ascending"),
    ("direct", dict(algo="direct"), "ascending"),
    ("ring rotated", dict(algo="ring", fuse=0, order="ring"), "ring"),
    ("two-level 4x2", dict(algo="two_level", group_size=4, fuse=0), "two_level"),
    ("two-level fused", dict(algo="two_level", group_size=4), "two_level"),
    ("rhd butterfly", dict(algo="rhd", order="halving", fuse=0), "halving"),
    ("rhd fused", dict(algo="rhd", order="halving"), "halving"),
]


@pytest.mark.parametrize("dt", ["bf16", "fp32", "int32", "fp16"])
@pytest.mark.parametrize("label,cfg,order", ALLREDUCE, ids=[a[0] for a in ALLREDUCE])
def test_allreduce_programs_in_random_orders(label, cfg, order, dt):
    P, N = 8, 1500
    x = inputs(P, N, dt, seed=10)
    with H.Comm(P, device=H.NO_DEVICE, **cfg, **SMALL) as c:
        H.hccl_allreduce(c.handle, fake(P, 1 << 40), fake(P, 1 << 44), N, dt)
        image = c.program_image()
    want = oracle.allreduce_ordered(x, dt, order=order, group=cfg.get("group_size", 0), shard=shard(N, P))
    for seed in SEEDS:
        (got,) = run_program(image, list(x), [N * ES[dt]] * P, seed)
        check(got, want, dt)


@pytest.mark.parametrize("cfg,order", [(dict(algo="ring", fuse=0, requantize=1), "ascending"),
                                       (dict(algo="ring", fuse=0, order="ring", requantize=1), "ring"),
                                       (dict(algo="rhd", order="halving", fuse=0, requantize=1), "halving"),
                                       (dict(algo="two_level", group_size=2, fuse=0, requantize=1), "two_level")])
def test_requantised_partials_in_random_orders(cfg, order):
    P, N = 8, 1300
    x = inputs(P, N, "bf16", seed=11)
    with H.Comm(P, device=H.NO_DEVICE, **cfg, **SMALL) as c:
        H.hccl_allreduce(c.handle, fake(P, 1 << 40), fake(P, 1 << 44), N, "bf16")
        image = c.program_image()
    want = oracle.allreduce_ordered(x, "bf16", order=order, group=cfg.get("group_size", 0), shard=shard(N, P),
                                    requant=True)
    for seed in SEEDS:
        (got,) = run_program(image, list(x), [N * 2] * P, seed)
        check(got, want, "bf16")


@pytest.mark.parametrize("op", ["max", "min"])
def test_max_min_ring_in_random_orders(op):
    P, N = 5, 1111
    x = inputs(P, N, "fp32", seed=12)
    x[1, ::7] = np.nan
    with H.Comm(P, device=H.NO_DEVICE, algo="ring", fuse=0, **SMALL) as c:
        H.hccl_allreduce(c.handle, fake(P, 1 << 40), fake(P, 1 << 44), N, "fp32", op)
        image = c.program_image()
    want = oracle.allreduce(x, "fp32", op=op)
    for seed in SEEDS:
        (got,) = run_program(image, list(x), [N * 4] * P, seed)
        for r in range(P):
            g, w = got[r].view(np.float32), want[r]
            assert np.array_equal(np.isnan(g), np.isnan(w)) and np.array_equal(g[~np.isnan(g)], w[~np.isnan(w)])


@pytest.mark.parametrize("cfg,order", [(dict(algo="ring", fuse=0), "ascending"), (dict(algo="ring"), "ascending"),
                                       (dict(algo="ring", fuse=0, order="ring"), "ring"),
                                       (dict(algo="rhd", order="halving", fuse=0), "halving")])
def test_reduce_scatter_programs_in_random_orders(cfg, order):
    P, M = 4, 900
    x = inputs(P, P * M, "bf16", seed=13)
    with H.Comm(P, device=H.NO_DEVICE, **cfg, **SMALL) as c:
        H.hccl_reduce_scatter(c.handle, fake(P, 1 << 40), fake(P, 1 << 44), M, "bf16")
        image = c.program_image()
    want = oracle.reduce_scatter_ordered(x, "bf16", order=order)
    for seed in SEEDS:
        (got,) = run_program(image, list(x), [M * 2] * P, seed)
        check(got, want, "bf16")


@pytest.mark.parametrize("cfg", [dict(algo="ring", fuse=0), dict(algo="ring"), dict(algo="rhd", fuse=0),
                                 dict(algo="direct")])
def test_allgather_programs_in_random_orders(cfg):
    P, M = 8, 700
    x = inputs(P, M, "fp32", seed=14)
    with H.Comm(P, device=H.NO_DEVICE, **cfg, **SMALL) as c:
        H.hccl_allgather(c.handle, fake(P, 1 << 40), fake(P, 1 << 44), M, "fp32")
        image = c.program_image()
    want = oracle.allgather(x)
    for seed in SEEDS:
        (got,) = run_program(image, list(x), [P * M * 4] * P, seed)
        check(got, want, "fp32")


def test_alltoallv_program_with_split_pieces_in_random_orders():
    P = 6
    counts = zipf_counts(P, 300, 1.1, seed=15)
    lay = alltoallv_layout(counts, 7)
    rows = [normal_bf16(1, int(lay["send_len"][s]), seed=16 + s)[0] for s in range(P)]
    with H.Comm(P, device=H.NO_DEVICE, chunk_bytes=256) as c:
        H.hccl_alltoallv(c.handle, fake(P, 1 << 40), lay["sendcounts"], lay["sdispls"], fake(P, 1 << 44),
                         lay["recvcounts"], lay["rdispls"], "bf16")
        image = c.program_image()
        assert c.last_program()["num_descs"] > P * P      # blocks were split into pieces
    want = [np.zeros(int(lay["recv_len"][d]), np.uint16) for d in range(P)]
    oracle.alltoallv(rows, lay["sendcounts"], lay["sdispls"], want, lay["recvcounts"], lay["rdispls"])
    for seed in SEEDS:
        (got,) = run_program(image, rows, [int(n) * 2 for n in lay["recv_len"]], seed)
        check(got, want, "bf16")


@pytest.mark.parametrize("phases", ["one", "auto"])
def test_group_of_dependent_programs_in_random_orders(phases):
    P = 4
    xa = inputs(P, 2000, "bf16", seed=17)
    xb = inputs(P, P * 600, "fp32", seed=18)
    xc = inputs(P, 333, "bf16", seed=19)
    with H.Comm(P, device=H.NO_DEVICE, algo="ring", fuse=0, phases=phases, **SMALL) as c:
        with c.group():
            H.hccl_allreduce(c.handle, fake(P, 1 << 40), fake(P, 2 << 40), 2000, "bf16")
            H.hccl_reduce_scatter(c.handle, fake(P, 3 << 40), fake(P, 4 << 40), 600, "fp32")
            H.hccl_allgather(c.handle, fake(P, 5 << 40), fake(P, 6 << 40), 333, "bf16")
        image = c.program_image()
        info = c.last_program()
        assert info["collective"] == -1
        # one launch waiting tile by tile, or the three calls' hops level by level (the
        # all-reduce has the most: 2 reduce hops + 3 forwarding hops after its first step)
        assert (info["num_deps"] > 0 and info["num_phases"] == 1) if phases == "one" else \
            (info["num_deps"] == 0 and info["num_phases"] == 6)
    layout = [(P, list(xa), [2000 * 2] * P), (P, list(xb), [600 * 4] * P), (P, list(xc), [P * 333 * 2] * P)]
    for seed in SEEDS:
        ga, gb, gc = run_program(image, None, None, seed, group_layout=layout)
        check(ga, oracle.allreduce(xa, "bf16"), "bf16")
        check(gb, oracle.reduce_scatter(xb, "fp32"), "fp32")
        check(gc, oracle.allgather(xc), "bf16")


def test_image_is_empty_before_any_program():
    with H.Comm(2, device=H.NO_DEVICE) as c:
        assert c.program_image() == b""


@pytest.mark.parametrize("cfg,order", [(dict(algo="two_level", group_size=4), "two_level"),
                                       (dict(algo="ring"), "ascending"),
                                       (dict(algo="two_level", group_size=16), "two_level")],
                         ids=["two-level 4x4", "ring", "two-level 1x16"])
def test_wide_reduction_with_split_copies_in_random_orders(cfg, order):
    """16 ranks: every reduction has 16 sources, so under phases=levels its result is written
    once and copied to the other 15 ranks by a second phase."""
    P, N = 16, 2500
    x = inputs(P, N, "bf16", seed=21)
    with H.Comm(P, device=H.NO_DEVICE, phases="levels", **cfg, **SMALL) as c:
        H.hccl_allreduce(c.handle, fake(P, 1 << 40), fake(P, 1 << 44), N, "bf16")
        image = c.program_image()
        info = c.last_program()
    assert info["num_phases"] == 2 and info["num_deps"] == 0
    assert info["bytes_read"] == P * N * 2 + N * 2 and info["bytes_written"] == P * N * 2
    want = oracle.allreduce_ordered(x, "bf16", order=order, group=cfg.get("group_size", 0), shard=shard(N, P))
    for seed in SEEDS:
        (got,) = run_program(image, list(x), [N * 2] * P, seed)
        check(got, want, "bf16")
