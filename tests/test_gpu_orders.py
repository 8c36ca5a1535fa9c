"""GPU parity for the ring order, the recursive-halving order and re-quantised partials.

Each schedule that can produce an order (one-shot DIRECT, RING chains, RHD butterfly), fused
and unfused, must give the bits the oracle computes for that order, through the C-ABI.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import Guarded, first_mismatch, same_bits, to_device
from test_gpu_parity import inputs

pytestmark = pytest.mark.gpu


def lib_shard(N, P):
    # the all-reduce shard of the ring order: ceil(N / P) rounded up to 64 elements
    q = -(-N // P)
    return -(-q // 64) * 64


def run_ar(P, N, dt, order, requant, **cfg):
    x = inputs(P, N, dt, seed=P * 7 + N)
    print(f"allreduce order={order} requant={requant} P={P} N={N} dt={dt} cfg={cfg}", flush=True)
    with H.Comm(P, device=0, order=order, requantize=int(requant), **cfg) as c:
        send = [to_device(x[r], dt) for r in range(P)]
        outs = [Guarded(N, dt) for _ in range(P)]
        H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, dt)
        torch.cuda.synchronize()
        assert c.async_error() == 0
        info = c.last_program()
    want = oracle.allreduce_ordered(x, dt, order="ring" if order == "ring" else
                                    ("halving" if order == "halving" else "ascending"),
                                    shard=lib_shard(N, P), requant=requant)
    for r in range(P):
        got = outs[r].result()
        assert same_bits(got, want[r], dt), f"rank {r}: {first_mismatch(got, want[r])}"
        assert outs[r].guards_intact()
    return info


def run_rs(P, M, dt, order, requant, **cfg):
    x = inputs(P, P * M, dt, seed=P * 11 + M)
    print(f"reduce_scatter order={order} requant={requant} P={P} M={M} dt={dt} cfg={cfg}", flush=True)
    with H.Comm(P, device=0, order=order, requantize=int(requant), **cfg) as c:
        send = [to_device(x[r], dt) for r in range(P)]
        outs = [Guarded(M, dt) for _ in range(P)]
        H.hccl_reduce_scatter(c.handle, send, [o.view for o in outs], M, dt)
        torch.cuda.synchronize()
        assert c.async_error() == 0
    want = oracle.reduce_scatter_ordered(x, dt, order=order, requant=requant)
    for r in range(P):
        got = outs[r].result()
        assert same_bits(got, want[r], dt), f"rank {r}: {first_mismatch(got, want[r])}"
        assert outs[r].guards_intact()


SMALL = dict(chunk_bytes=4096, tile_bytes=4096)


@pytest.mark.parametrize("dt", ["bf16", "fp32", "fp16"])
@pytest.mark.parametrize("P", [2, 3, 8])
@pytest.mark.parametrize("algo,fuse", [("direct", 1), ("ring", 1), ("ring", 0)])
@pytest.mark.parametrize("requant", [False, True])
def test_ring_order(dt, P, algo, fuse, requant):
    run_ar(P, 10007, dt, "ring", requant, algo=algo, fuse=fuse, **SMALL)
    run_rs(P, 2001, dt, "ring", requant, algo=algo, fuse=fuse, **SMALL)


@pytest.mark.parametrize("dt", ["bf16", "fp32", "int32"])
@pytest.mark.parametrize("P", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("algo,fuse", [("direct", 1), ("rhd", 1), ("rhd", 0)])
@pytest.mark.parametrize("requant", [False, True])
def test_halving_order(dt, P, algo, fuse, requant):
    info = run_ar(P, 9001, dt, "halving", requant, algo=algo, fuse=fuse, **SMALL)
    if fuse and P > 1:
        assert info["num_deps"] == 0
    run_rs(P, 1501, dt, "halving", requant, algo=algo, fuse=fuse, **SMALL)


def test_halving_order_with_64_sources_fills_the_tree():
    run_ar(64, 4099, "bf16", "halving", False, algo="direct")
    run_ar(64, 4099, "bf16", "halving", True, algo="rhd", fuse=1, chunk_bytes=4096)


@pytest.mark.parametrize("fuse", [0, 1])
def test_rhd_allgather(fuse):
    P, M = 8, 3001
    x = inputs(P, M, "bf16", 5)
    with H.Comm(P, device=0, algo="rhd", fuse=fuse, **SMALL) as c:
        send = [to_device(x[r], "bf16") for r in range(P)]
        outs = [Guarded(P * M, "bf16") for _ in range(P)]
        H.hccl_allgather(c.handle, send, [o.view for o in outs], M, "bf16")
        torch.cuda.synchronize()
        assert c.async_error() == 0
    want = oracle.allgather(x)
    for r in range(P):
        assert np.array_equal(outs[r].result(), want[r]) and outs[r].guards_intact()


@pytest.mark.parametrize("fuse", [0, 1])
def test_rhd_in_place_allreduce(fuse):
    P, N = 8, 20000
    x = inputs(P, N, "fp32", 6)
    with H.Comm(P, device=0, algo="rhd", order="halving", fuse=fuse, **SMALL) as c:
        bufs = [Guarded(N, "fp32", fill=x[r]) for r in range(P)]
        H.hccl_allreduce(c.handle, [b.view for b in bufs], [b.view for b in bufs], N, "fp32")
        torch.cuda.synchronize()
        assert c.async_error() == 0
    want = oracle.allreduce_ordered(x, "fp32", order="halving")
    for r in range(P):
        assert same_bits(bufs[r].result(), want[r], "fp32") and bufs[r].guards_intact()


@pytest.mark.parametrize("fuse", [0, 1])
def test_requantized_ascending_chains(fuse):
    run_ar(8, 30011, "bf16", "ascending", True, algo="ring", fuse=fuse, **SMALL)
    run_rs(8, 3001, "fp16", "ascending", True, algo="ring", fuse=fuse, **SMALL)


def test_two_level_with_requantized_partials():
    P, L, N = 16, 4, 8000
    x = inputs(P, N, "bf16", 8)
    for fuse in (0, 1):
        with H.Comm(P, device=0, algo="two_level", group_size=L, fuse=fuse, requantize=1, **SMALL) as c:
            send = [to_device(x[r], "bf16") for r in range(P)]
            outs = [Guarded(N, "bf16") for _ in range(P)]
            H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, "bf16")
            torch.cuda.synchronize()
        want = oracle.allreduce_ordered(x, "bf16", order="two_level", group=L, requant=True)
        for r in range(P):
            assert same_bits(outs[r].result(), want[r], "bf16"), f"fuse={fuse} rank {r}"
