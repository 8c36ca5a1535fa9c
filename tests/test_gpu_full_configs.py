"""Parity at the full benchmark sizes.

Every output element is compared with the oracle (the oracle finishes each of these in
seconds on the host). Inputs come from the same seeded generators as bench.py: host
generators for the small configurations, the seeded device generator for the large ones
(copied back to the host for the oracle). The AllToAllv configuration is run both in the
form bench.py times (rows and ids recorded in one group: one program, one launch, whose copy
steps have 4096-element bf16 tiles beside 2048-element int32 tiles) and as two launches.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import first_mismatch, same_bits, to_device, to_host
from workloads import (alltoallv_layout, device_normal_bf16, row_ids_int32, uniform_f32,
                       zipf_counts)

pytestmark = pytest.mark.gpu
MiB = 1 << 20


def _host_bits(tensors, dt):
    return np.stack([to_host(t, dt) for t in tensors])


def test_allreduce_ring_p4_fp32_full():
    P, N = 4, 1 << 20
    print("full config: allreduce ring P=4 N=2^20 fp32 chunk 64 KiB", flush=True)
    x = uniform_f32(P, N, seed=0)
    send = [to_device(x[r], "fp32") for r in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    with H.Comm(P, device=0, algo="ring", chunk_bytes=64 * 1024) as c:
        c.allreduce(send, recv)
        torch.cuda.synchronize()
        assert c.async_error() == 0
    want = oracle.allreduce(x, "fp32")
    for r in range(P):
        got = to_host(recv[r], "fp32")
        assert same_bits(got, want[r], "fp32", nan_equal=False), f"rank {r}: {first_mismatch(got, want[r])}"


def _alltoallv_rows_ids_oracle(send_rows, id_vals, rows, ids, P):
    host_rows = [to_host(t, "bf16") for t in send_rows]
    want_rows = [np.zeros(int(rows["recv_len"][d]), np.uint16) for d in range(P)]
    oracle.alltoallv(host_rows, rows["sendcounts"], rows["sdispls"], want_rows, rows["recvcounts"], rows["rdispls"])
    want_ids = [np.zeros(int(ids["recv_len"][d]), np.int32) for d in range(P)]
    oracle.alltoallv([id_vals[s] for s in range(P)], ids["sendcounts"], ids["sdispls"], want_ids,
                     ids["recvcounts"], ids["rdispls"])
    return want_rows, want_ids


def test_alltoallv_zipf_p8_rows_and_ids_grouped_one_launch_as_benchmarked():
    """The timed headline step: rows and ids as one group, compiled into one program whose row
    steps keep 8 KiB (4096-element) tiles beside the ids' 2048-element tiles, one launch."""
    P, R, D = 8, 1 << 18, 128
    print("full config: alltoallv P=8 2^18 rows x 128 bf16 Zipf(1.1) + int32 ids, one grouped launch", flush=True)
    counts = zipf_counts(P, R, 1.1, seed=0)
    rows, ids = alltoallv_layout(counts, D), alltoallv_layout(counts, 1)
    send_rows = device_normal_bf16(P, R * D, seed=0)
    id_vals = row_ids_int32(P, R, seed=1)
    send_ids = [to_device(id_vals[s], "int32") for s in range(P)]
    # receive buffers start from a poison pattern: a range the launch skipped would show
    recv_rows = [torch.full((int(rows["recv_len"][d]),), -7.0, dtype=torch.bfloat16, device="cuda:0")
                 for d in range(P)]
    recv_ids = [torch.full((int(ids["recv_len"][d]),), -5, dtype=torch.int32, device="cuda:0") for d in range(P)]
    with H.Comm(P, device=0) as c:
        for _ in range(2):   # the second launch reuses the cached program, as the timed steps do
            with c.group():
                c.alltoallv(send_rows, rows["sendcounts"], rows["sdispls"], recv_rows, rows["recvcounts"],
                            rows["rdispls"])
                c.alltoallv(send_ids, ids["sendcounts"], ids["sdispls"], recv_ids, ids["recvcounts"], ids["rdispls"])
        torch.cuda.synchronize()
        info = c.last_program()
        assert c.async_error() == 0
    assert info["collective"] == -1 and info["cache_hit"] == 1 and info["inline_launch"] == 0
    assert (info["step_tile_min"], info["step_tile_max"]) == (2048, 4096), info
    assert info["bytes_read"] == info["bytes_written"] == int(rows["sendcounts"].sum()) * 2 + int(
        ids["sendcounts"].sum()) * 4
    want_rows, want_ids = _alltoallv_rows_ids_oracle(send_rows, id_vals, rows, ids, P)
    for d in range(P):
        assert np.array_equal(to_host(recv_rows[d], "bf16"), want_rows[d]), f"rows at destination {d}"
        assert np.array_equal(to_host(recv_ids[d], "int32"), want_ids[d]), f"ids at destination {d}"
    print(f"grouped launch: {info['num_descs']} steps, {info['num_tiles']} tiles, {info['workers']} wavefronts",
          flush=True)


def test_alltoallv_zipf_p8_embedding_rows_and_ids_full_as_two_launches():
    P, R, D = 8, 1 << 18, 128
    print("full config: alltoallv P=8 2^18 rows x 128 bf16 Zipf(1.1) + int32 ids, two launches", flush=True)
    counts = zipf_counts(P, R, 1.1, seed=0)
    rows, ids = alltoallv_layout(counts, D), alltoallv_layout(counts, 1)
    send_rows = device_normal_bf16(P, R * D, seed=0)
    id_vals = row_ids_int32(P, R, seed=1)
    send_ids = [to_device(id_vals[s], "int32") for s in range(P)]
    recv_rows = [torch.empty(int(rows["recv_len"][d]), dtype=torch.bfloat16, device="cuda:0") for d in range(P)]
    recv_ids = [torch.empty(int(ids["recv_len"][d]), dtype=torch.int32, device="cuda:0") for d in range(P)]
    with H.Comm(P, device=0) as c:
        c.alltoallv(send_rows, rows["sendcounts"], rows["sdispls"], recv_rows, rows["recvcounts"], rows["rdispls"])
        c.alltoallv(send_ids, ids["sendcounts"], ids["sdispls"], recv_ids, ids["recvcounts"], ids["rdispls"])
        torch.cuda.synchronize()
        assert c.async_error() == 0
    want_rows, want_ids = _alltoallv_rows_ids_oracle(send_rows, id_vals, rows, ids, P)
    for d in range(P):
        assert np.array_equal(to_host(recv_rows[d], "bf16"), want_rows[d]), f"rows at destination {d}"
        assert np.array_equal(to_host(recv_ids[d], "int32"), want_ids[d]), f"ids at destination {d}"
    # every received row still carries its id: the two calls used one split
    total = sum(int(n) for n in rows["recv_len"]) * 2
    assert total == 2 * P * R * D


def test_reduce_scatter_ring_p8_256mib_bf16_full():
    P = 8
    M = (256 * MiB // 2) // P
    print("full config: reduce_scatter ring P=8 256 MiB/rank bf16 chunk 1 MiB", flush=True)
    send = device_normal_bf16(P, P * M, std=0.02, seed=0)
    recv = [torch.empty(M, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
    with H.Comm(P, device=0, algo="ring", chunk_bytes=MiB) as c:
        c.reduce_scatter(send, recv)
        torch.cuda.synchronize()
        assert c.async_error() == 0
    x = _host_bits(send, "bf16")
    del send
    want = oracle.reduce_scatter(x, "bf16")
    for r in range(P):
        got = to_host(recv[r], "bf16")
        assert np.array_equal(got, want[r]), f"rank {r}: {first_mismatch(got, want[r])}"


def test_two_level_allreduce_p64_32mib_bf16_full_and_ulp_distance_to_flat_order():
    P, L = 64, 8
    N = 32 * MiB // 2
    print("full config: allreduce two-level P=64 (8x8) 32 MiB/rank bf16", flush=True)
    send = device_normal_bf16(P, N, seed=0)
    recv = [torch.empty(N, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
    with H.Comm(P, device=0, algo="two_level", group_size=L) as c:
        c.allreduce(send, recv)
        torch.cuda.synchronize()
        assert c.async_error() == 0
    for r in range(1, P):
        assert torch.equal(recv[r].view(torch.int16), recv[0].view(torch.int16)), f"rank {r} differs from rank 0"
    x = _host_bits(send, "bf16")
    del send
    got = to_host(recv[0], "bf16")
    del recv
    torch.cuda.empty_cache()
    # the oracle's all-reduce writes every rank's copy; one rank's worth of columns at a time
    cols = 1 << 21
    ulps = []
    for lo in range(0, N, cols):
        blk = np.ascontiguousarray(x[:, lo:lo + cols])
        tree = oracle.allreduce(blk, "bf16", group=L)[0]
        assert np.array_equal(got[lo:lo + cols], tree), f"columns {lo}..: {first_mismatch(got[lo:lo + cols], tree)}"
        flat = oracle.allreduce(blk, "bf16")[0]
        # distance in bf16 units in the last place between the two fold orders
        a = oracle.bf16_to_f32(tree).astype(np.float64)
        b = oracle.bf16_to_f32(flat).astype(np.float64)
        ulp = np.spacing(np.maximum(np.abs(a), np.abs(b)).astype(np.float32)).astype(np.float64) * 2 ** 16
        ulps.append(np.abs(a - b) / ulp)
    d = np.concatenate(ulps)
    print(f"two-level vs flat order: max {d.max():.2f} bf16 ulp, {(d > 1).sum()} of {d.size} elements above 1 ulp, "
          f"{(d > 0).sum()} differ", flush=True)
    assert d.max() <= 2.0


def test_latency_config_allreduce_p8_64kib_fp32_full():
    P, N = 8, 1 << 14
    print("full config: allreduce direct P=8 64 KiB/rank fp32", flush=True)
    x = uniform_f32(P, N, seed=5)
    send = [to_device(x[r], "fp32") for r in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    with H.Comm(P, device=0, algo="direct") as c:
        for _ in range(3):
            c.allreduce(send, recv)
        torch.cuda.synchronize()
        assert c.async_error() == 0
    want = oracle.allreduce(x, "fp32")
    for r in range(P):
        assert same_bits(to_host(recv[r], "fp32"), want[r], "fp32", nan_equal=False), f"rank {r}"
