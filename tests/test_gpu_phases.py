"""GPU parity of phased programs: the wide reductions whose results a second launch copies to
the other ranks, and dependent schedules run one launch per dependency level, against the
oracle bit for bit (ragged sizes, every element type, MAX / MIN, in place)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import Guarded, first_mismatch, same_bits, to_device
from test_gpu_parity import inputs, run_allreduce

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt", ["bf16", "fp32", "fp16", "int32"])
@pytest.mark.parametrize("P,L", [(16, 4), (32, 8), (64, 8), (16, 16)])
def test_two_level_with_split_copies(P, L, dt):
    """phases=levels forces the split at a small size: 64-, 32- or 16-source reductions write
    each sub-shard once, a second launch copies it to the other ranks (8 KiB and larger tiles,
    a ragged tail)."""
    info = run_allreduce(P, 30011, dt, algo="two_level", group_size=L, phases="levels", seed=P + L)
    assert info["num_phases"] == 2 and info["num_deps"] == 0 and info["max_srcs"] == P
    assert info["bytes_read"] == (P + 1) * 30011 * {"bf16": 2, "fp16": 2, "fp32": 4, "int32": 4}[dt]


@pytest.mark.parametrize("op", ["max", "min"])
@pytest.mark.parametrize("dt", ["fp32", "bf16"])
def test_split_copies_max_min(op, dt):
    info = run_allreduce(16, 9001, dt, op=op, algo="two_level", group_size=4, phases="levels", seed=3)
    assert info["num_phases"] == 2


@pytest.mark.parametrize("P", [16, 24])
def test_flat_ring_with_split_copies(P):
    """The fused ring of 16 or 24 ranks: one P-source reduction per chunk into its owner, then
    the owner's copy to the other P-1 ranks (the chained hops merged into one copy)."""
    info = run_allreduce(P, 50001, "bf16", algo="ring", phases="levels", chunk_bytes=16384, seed=P)
    assert info["num_phases"] == 2 and info["num_deps"] == 0


def test_split_copies_in_place():
    P, N = 16, 20011
    info = run_allreduce(P, N, "bf16", in_place=True, algo="two_level", group_size=4, phases="levels", seed=5)
    assert info["num_phases"] == 2


@pytest.mark.parametrize("dt", ["fp16", "int32", "fp32"])
@pytest.mark.parametrize("P", [3, 5, 8])
def test_unfused_reduce_scatter_and_allgather_level_by_level(P, dt):
    """Ring reduce-scatter and all-gather with every hop a step of its own, one launch per
    hop, ragged sizes."""
    M = 7777
    x = inputs(P, P * M, dt, seed=40 + P)
    y = inputs(P, M, dt, seed=50 + P)
    print(f"levels: reduce_scatter and allgather P={P} M={M} dt={dt}", flush=True)
    with H.Comm(P, device=0, algo="ring", fuse=0, chunk_bytes=4096, tile_bytes=4096) as c:
        send = [to_device(x[r], dt) for r in range(P)]
        rs = [Guarded(M, dt) for _ in range(P)]
        H.hccl_reduce_scatter(c.handle, send, [o.view for o in rs], M, dt)
        rs_info = c.last_program()
        ysend = [to_device(y[r], dt) for r in range(P)]
        ag = [Guarded(P * M, dt) for _ in range(P)]
        H.hccl_allgather(c.handle, ysend, [o.view for o in ag], M, dt)
        ag_info = c.last_program()
        torch.cuda.synchronize()
        assert c.async_error() == 0
    assert rs_info["num_phases"] == P - 1 and rs_info["num_deps"] == 0
    assert ag_info["num_phases"] == P and ag_info["num_deps"] == 0
    want_rs, want_ag = oracle.reduce_scatter(x, dt), oracle.allgather(y)
    for r in range(P):
        got = rs[r].result()
        assert same_bits(got, want_rs[r], dt), f"reduce_scatter rank {r}: {first_mismatch(got, want_rs[r])}"
        got = ag[r].result()
        assert same_bits(got, want_ag[r], dt), f"allgather rank {r}: {first_mismatch(got, want_ag[r])}"
        assert rs[r].guards_intact() and ag[r].guards_intact()


def test_phased_program_repeated_on_two_streams():
    """A four-level program launched again and again on two streams: every launch right."""
    P, N = 16, 40000
    x = inputs(P, N, "fp32", 61)
    want = oracle.allreduce(x, "fp32", group=4)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    print("levels: unfused two-level on two streams", flush=True)
    with H.Comm(P, device=0, algo="two_level", group_size=4, fuse=0, chunk_bytes=16384) as c:
        send = [to_device(x[r], "fp32") for r in range(P)]
        o1 = [Guarded(N, "fp32") for _ in range(P)]
        o2 = [Guarded(N, "fp32") for _ in range(P)]
        torch.cuda.synchronize()
        for _ in range(3):
            H.hccl_allreduce(c.handle, send, [o.view for o in o1], N, "fp32", stream=s1)
            H.hccl_allreduce(c.handle, send, [o.view for o in o2], N, "fp32", stream=s2)
        torch.cuda.synchronize()
        assert c.async_error() == 0
        assert c.last_program()["num_phases"] == 4
    for r in range(P):
        assert same_bits(o1[r].result(), want[r], "fp32") and same_bits(o2[r].result(), want[r], "fp32")
