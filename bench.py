#!/usr/bin/env python3
"""Benchmark of the HCCL copy/reduce hot path on one MI355X.

A step is one AllToAllv of recommendation-shaped data over P = 8 virtual ranks: every rank
sends 2^18 embedding rows (128 bf16 = 256 B each, 64 MiB) split across destinations by a
Zipf(1.1) law, then the int32 row ids ride along in a second call. The metric is effective
HBM GB/s = algorithmic bytes / time, algorithmic bytes = 2 x payload (each byte read once,
written once). Inputs are resident in HBM before timing starts.

The same JSON line carries the roofline of the dominant kernel (the embedding-row launch,
timed with HIP events on its stream), the CPU oracle timed on the host, and the other
collective workloads measured the same way (ring all-reduce, ring reduce-scatter, two-level
all-reduce, small-message latency, GEMM overlap on a CU-masked stream).

python bench.py [--gpus 1] [--steps K] [--warmup W] [--headline-only] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MiB = 1 << 20


def _log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _time_events(fn, iters: int, stream=None):
    """Runs fn() iters times back to back; returns per-iteration ms from one event pair."""
    import torch

    s = stream or torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record(s)
    for _ in range(iters):
        fn()
    b.record(s)
    b.synchronize()
    return a.elapsed_time(b) / iters


# ------------------------------------------------------------------------- headline
def alltoallv_workload(device):
    import numpy as np

    from workloads import alltoallv_layout, device_normal_bf16, row_ids_int32, zipf_counts

    P, R, D = 8, 1 << 18, 128
    counts = zipf_counts(P, R, 1.1, seed=0)
    rows = alltoallv_layout(counts, D)
    ids = alltoallv_layout(counts, 1)
    t0 = time.time()
    send_rows = device_normal_bf16(P, R * D, seed=0, device=device)   # each rank sends exactly R rows
    id_vals = row_ids_int32(P, R, seed=1)
    _log(f"alltoallv inputs generated in {time.time() - t0:.1f}s")
    return {"P": P, "R": R, "D": D, "counts": counts, "rows": rows, "ids": ids,
            "send_rows": send_rows, "id_vals": id_vals}


def run_headline(args, device):
    """Times K steps of the grouped AllToAllv (rows + ids in one work packet, one launch).
    One pair of HIP events on the launch stream brackets the K back-to-back launches: their
    span / K is the average launch duration (the gaps between launches included), and nothing
    is recorded between steps, so the host-timed steps carry no instrumentation. Also times
    the two calls issued separately (before the grouped steps, so that the receive buffers
    hold the timed steps' results for the CPU baseline's check)."""
    import torch

    import paper_2608_00358_amd as H

    w = alltoallv_workload(device)
    P = w["P"]
    rows, ids = w["rows"], w["ids"]
    send_rows = w["send_rows"]
    send_ids = [torch.from_numpy(w["id_vals"][s].copy()).to(device) for s in range(P)]
    recv_rows = [torch.empty(int(rows["recv_len"][d]), dtype=torch.bfloat16, device=device) for d in range(P)]
    recv_ids = [torch.empty(int(ids["recv_len"][d]), dtype=torch.int32, device=device) for d in range(P)]
    row_bytes = int(rows["sendcounts"].sum()) * 2
    id_bytes = int(ids["sendcounts"].sum()) * 4
    comm = H.Comm(P, device=0)
    rows_call = comm.bind_alltoallv(send_rows, rows["sendcounts"], rows["sdispls"], recv_rows,
                                    rows["recvcounts"], rows["rdispls"])
    ids_call = comm.bind_alltoallv(send_ids, ids["sendcounts"], ids["sdispls"], recv_ids,
                                   ids["recvcounts"], ids["rdispls"])

    def step():
        H.hccl_group_start(comm.handle)
        rows_call()
        ids_call()
        H.hccl_group_end(comm.handle)

    algo_step = 2 * (row_bytes + id_bytes)
    # the same two collectives as two launches (timed first: the receive buffers must hold
    # what the timed grouped steps wrote)
    separate = {}
    if not args.headline_only:
        for _ in range(3):
            rows_call()
            ids_call()
        ms_rows = _time_events(rows_call, args.steps)
        ms_sep = _time_events(lambda: (rows_call(), ids_call()), args.steps)
        separate = {"rows_launch_us": ms_rows * 1e3, "rows_launch_gbs": 2 * row_bytes / (ms_rows * 1e-3) / 1e9,
                    "two_launch_step_us": ms_sep * 1e3,
                    "two_launch_step_gbs": algo_step / (ms_sep * 1e-3) / 1e9}

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    info_step = comm.last_program()
    # poison the receive buffers: after the timed steps they hold only what those steps wrote
    for t in recv_rows:
        t.fill_(float("nan"))
    for t in recv_ids:
        t.fill_(-1)

    s = torch.cuda.current_stream()
    first = torch.cuda.Event(enable_timing=True)
    last = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    first.record(s)
    for _ in range(args.steps):
        step()
    last.record(s)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    if comm.async_error() != 0:
        raise RuntimeError(H.hccl_get_last_error())
    ms_step = elapsed * 1e3 / args.steps
    launch_ms = first.elapsed_time(last) / args.steps
    # host cost of re-enqueueing the cached work packet (group start, two calls, group end:
    # four ctypes calls and one launch); the GPU is left to drain afterwards
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    host_us = (time.perf_counter() - t0) * 1e6 / args.steps
    torch.cuda.synchronize()

    recv_counts = w["counts"].sum(axis=0)
    w.update({"send_ids": send_ids, "recv_rows": recv_rows, "recv_ids": recv_ids})
    result = {
        "ms_per_step": ms_step,
        "value": algo_step / (ms_step * 1e-3) / 1e9,
        "launch_ms": launch_ms,
        "algo_bytes_step": algo_step,
        "recv_imbalance": float(recv_counts.max() / recv_counts.mean()),
        "program": info_step,
        "separate_calls": separate,
        "host_enqueue_us": host_us,
    }
    comm.close()
    return result, w


def _extra(name, fn):
    """Runs one secondary measurement; an error in it is recorded in its place instead of
    costing the headline line (a GPU fault still ends the process)."""
    try:
        return fn()
    except Exception as e:  # noqa: BLE001
        _log(f"{name} failed: {type(e).__name__}: {e}")
        return {"error": f"{type(e).__name__}: {e}"}


# --------------------------------------------------------------------- other configs
def bench_allreduce_ring_c1(device, iters=200, cold_sets=40):
    """All-reduce P=4 x 2^20 fp32 U[-1,1), ring reduce-scatter + all-gather, 64 KiB chunks."""
    import torch

    import paper_2608_00358_amd as H
    from workloads import uniform_f32

    P, N = 4, 1 << 20
    x = uniform_f32(P, N, seed=0)
    send = [torch.from_numpy(x[r].copy()).to(device) for r in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device=device) for _ in range(P)]
    algo = 2 * P * N * 4
    out = {}
    def warmed(call):
        call()   # the first call compiles and uploads the program: outside the timing
        torch.cuda.synchronize()
        return call

    with H.Comm(P, device=0, algo="ring", chunk_bytes=64 * 1024) as c:
        ms = _time_events(warmed(c.bind_allreduce(send, recv)), iters)
        info = c.last_program()
        out["warm_us"] = ms * 1e3
        out["warm_gbs"] = algo / (ms * 1e-3) / 1e9
        # cold: rotate through enough buffer sets to defeat the 256 MiB infinity cache
        sets = [([torch.empty(N, dtype=torch.float32, device=device).copy_(t) for t in send],
                 [torch.empty(N, dtype=torch.float32, device=device) for _ in range(P)]) for _ in range(cold_sets)]
        calls = [c.bind_allreduce(s, r) for s, r in sets]
        k = [0]

        def cold():
            calls[k[0] % cold_sets]()
            k[0] += 1

        ms = _time_events(cold, iters)
        out["cold_us"] = ms * 1e3
        out["cold_gbs"] = algo / (ms * 1e-3) / 1e9
        # the same program with every ring step as its own dependent descriptor: one launch per
        # hop (the default), and one launch whose steps wait for each other tile by tile
        for phases in ("auto", "one"):
            c.set_config(algo="ring", chunk_bytes=64 * 1024, fuse=0, phases=phases)
            ms = _time_events(warmed(c.bind_allreduce(send, recv)), iters)
            key = "unfused" if phases == "auto" else "unfused_one_launch"
            out[f"{key}_warm_us"] = ms * 1e3
            out[f"{key}_warm_gbs"] = algo / (ms * 1e-3) / 1e9
            out[f"{key}_launches"] = c.last_program()["num_phases"]
    out.update({"workload": "allreduce ring P=4 N=2^20 fp32 chunk=64KiB", "algo_bytes": algo,
                "descs": info["num_descs"], "tiles": info["num_tiles"], "compile_us": round(info["compile_us"], 1)})
    return out


def bench_reduce_scatter_c3(device, iters=20):
    """Reduce-scatter P=8 x 256 MiB bf16 N(0, 0.02), ascending fp32 fold, 1 MiB ring chunks."""
    import torch

    import paper_2608_00358_amd as H
    from workloads import device_normal_bf16

    P = 8
    M = (256 * MiB // 2) // P
    send = device_normal_bf16(P, P * M, std=0.02, seed=0, device=device)
    recv = [torch.empty(M, dtype=torch.bfloat16, device=device) for _ in range(P)]
    algo = (P + 1) * P * M * 2
    with H.Comm(P, device=0, algo="ring", chunk_bytes=MiB) as c:
        c.reduce_scatter(send, recv)
        ms = _time_events(lambda: c.reduce_scatter(send, recv), iters)
        info = c.last_program()
    res = {"workload": "reduce_scatter ring P=8 256MiB/rank bf16 chunk=1MiB", "us": ms * 1e3,
           "gbs": algo / (ms * 1e-3) / 1e9, "algo_bytes": algo, "descs": info["num_descs"],
           "compile_us": round(info["compile_us"], 1),
           "tiles": info["num_tiles"], "workers": info["workers"]}
    res["frac"] = res["gbs"] / HBM_PEAK_GBS
    return res, send, recv


def _bf16_ulp_distance(a, b):
    """Elementwise distance in bf16 units in the last place between two bf16 tensors (the
    encodings mapped to ordered integers: +0 and -0 coincide)."""
    import torch

    def ordered(t):
        u = t.view(torch.int16).to(torch.int32) & 0xFFFF
        mag = u & 0x7FFF
        return torch.where(u >= 0x8000, -mag, mag)

    return (ordered(a) - ordered(b)).abs()


def bench_forwarded_partials(device, iters=10):
    """The paper's forwarded-partial schedules (Section III-B-2 ring; recursive halving; Section
    II-A-2 per-result re-quantisation) on the reduce-scatter configuration (P=8, 256 MiB bf16 per
    rank, N(0, 0.02), 1 MiB chunks): time, effective GB/s, the schedule's own HBM bytes against
    the algorithmic bytes, and the numeric drift of each fold order against the ascending one
    (bf16 ulps; every schedule is bit-exact against the oracle in its own order)."""
    import torch

    import paper_2608_00358_amd as H
    from workloads import device_normal_bf16

    P = 8
    M = (256 * MiB // 2) // P
    send = device_normal_bf16(P, P * M, std=0.02, seed=0, device=device)
    algo = (P + 1) * P * M * 2
    variants = [
        ("ascending_ring_fused", dict(algo="ring")),
        ("ring_order_fused", dict(algo="ring", order="ring")),
        ("ring_order_forwarded_partials", dict(algo="ring", order="ring", fuse=0)),
        ("ring_order_forwarded_partials_one_launch", dict(algo="ring", order="ring", fuse=0, phases="one")),
        ("ring_order_forwarded_requantised", dict(algo="ring", order="ring", fuse=0, requantize=1)),
        ("halving_rhd_fused", dict(algo="rhd", order="halving")),
        ("halving_rhd_butterfly", dict(algo="rhd", order="halving", fuse=0)),
        ("halving_rhd_butterfly_one_launch", dict(algo="rhd", order="halving", fuse=0, phases="one")),
        ("halving_rhd_butterfly_requantised", dict(algo="rhd", order="halving", fuse=0, requantize=1)),
    ]
    ref = None
    out = {"workload": "reduce_scatter P=8 256MiB/rank bf16 N(0,0.02), 1 MiB chunks, fold orders and schedules",
           "algo_bytes": algo}
    for name, cfg in variants:
        recv = [torch.empty(M, dtype=torch.bfloat16, device=device) for _ in range(P)]
        with H.Comm(P, device=0, chunk_bytes=MiB, **cfg) as c:
            c.reduce_scatter(send, recv)
            ms = _time_events(lambda: c.reduce_scatter(send, recv), iters)
            info = c.last_program()
            if c.async_error() != 0:
                raise RuntimeError(H.hccl_get_last_error())
        sched = info["bytes_read"] + info["bytes_written"]
        res = {"us": round(ms * 1e3, 1), "gbs": round(algo / (ms * 1e-3) / 1e9, 1),
               "schedule_bytes": sched, "traffic_over_algorithmic": round(sched / algo, 4),
               "descs": info["num_descs"], "deps": info["num_deps"], "launches": info["num_phases"],
               "scratch_bytes": info["scratch_bytes"], "compile_us": round(info["compile_us"], 1)}
        if ref is None:
            ref = recv
        else:
            d = torch.cat([_bf16_ulp_distance(a, b) for a, b in zip(recv, ref)])
            res.update({"differ_from_ascending": int((d > 0).sum()), "above_1ulp": int((d > 1).sum()),
                        "max_ulp": int(d.max()), "mean_ulp": float(d.float().mean())})
        out[name] = res
        torch.cuda.synchronize()
    out["elements"] = P * M
    del send, ref
    torch.cuda.empty_cache()
    return out


def _stream_lib():
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_00358_amd", "lib", "libbench_stream.so"))
    lib.bench_stream.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64,
                                 ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p]
    lib.bench_stream_multi.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32,
                                       ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p]
    lib.bench_stream_reduce.argtypes = lib.bench_stream_multi.argtypes
    return lib


def _plain_reduce_ms(device, stream, region, streams=8, iters=3):
    """A plain bf16 sum of `streams` regions of `region` bytes into one (bench_stream.hip), on
    `stream`: the reduce-scatter's access pattern without the library, best of two grids (256
    workgroups, one wavefront per 4 KiB chunk)."""
    import torch

    lib = _stream_lib()
    a = torch.zeros(streams * region, dtype=torch.uint8, device=device)
    b = torch.empty(region, dtype=torch.uint8, device=device)
    best = float("inf")
    for bl in (256, region // 4096 // 4):
        def run():
            rc = lib.bench_stream_reduce(a.data_ptr(), b.data_ptr(), region, streams, 4096, bl, stream.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"bench_stream_reduce failed ({rc})")
        run()
        best = min(best, _time_events(run, iters, stream))
    del a, b
    return best


def bench_copy_ceiling(device, iters=20, nbytes=1 << 30):
    """What plain HIP kernels reach on this device (bench_stream.hip): a contiguous copy, a
    read-only and a write-only sweep of 1 GiB, read-only sweeps of 8 and 64 regions at the same
    offset, and a bf16 sum of 8 regions of 128 MiB into one (the reductions' patterns), each the
    best over grids of 1 024 and 2 048 workgroups and of one wavefront per chunk, chunks of 8 and
    32 KiB (4 KiB per region for the multi-region kernels) and 4 or 8 vectors per lane per step;
    and the library's own copy path on the same copy."""
    import torch

    lib = _stream_lib()
    a = torch.empty(nbytes, dtype=torch.uint8, device=device).fill_(7)
    b = torch.empty_like(a)
    st = torch.cuda.current_stream().cuda_stream
    out = {"workload": "1 GiB contiguous copy / read / write, 8 or 64 regions read, 8 x 128 MiB bf16 summed "
                       "into 128 MiB; non-temporal 16-byte loads"}

    def best_of(shapes, moved, launch, name):
        best = (0.0, None)
        for shape in shapes:
            def run():
                rc = launch(*shape)
                if rc != 0:
                    raise RuntimeError(f"{name} failed ({rc})")
            for _ in range(3):
                run()
            ms = _time_events(run, iters)
            best = max(best, (moved / (ms * 1e-3) / 1e9, shape), key=lambda x: x[0])
        return best

    for kind, name, moved in ((0, "copy", 2 * nbytes), (1, "read", nbytes), (2, "write", nbytes)):
        shapes = [(u, ch, bl) for u in (4, 8) for ch in (8192, 32768) for bl in (1024, 2048, nbytes // ch // 4)]
        gbs, (u, ch, bl) = best_of(shapes, moved, lambda u, ch, bl: lib.bench_stream(
            kind, u, a.data_ptr(), b.data_ptr(), nbytes, ch, bl, st), name)
        out[f"stream_{name}_gbs"] = round(gbs, 1)
        out[f"stream_{name}_shape"] = {"unroll": u, "chunk_bytes": ch, "blocks": bl}
    for streams in (8, 64):
        shapes = [(bl,) for bl in (256, 512, 1024, 2048, nbytes // streams // 4096 // 4)]
        gbs, (bl,) = best_of(shapes, nbytes, lambda bl: lib.bench_stream_multi(
            a.data_ptr(), b.data_ptr(), nbytes, streams, 4096, bl, st), f"read of {streams} regions")
        out[f"stream_read_{streams}_regions_gbs"], out[f"stream_read_{streams}_regions_blocks"] = round(gbs, 1), bl
    region = nbytes // 8
    shapes = [(bl,) for bl in (1024, 2048, 4096, region // 4096 // 4)]
    gbs, (bl,) = best_of(shapes, 9 * region, lambda bl: lib.bench_stream_reduce(
        a.data_ptr(), b.data_ptr(), region, 8, 4096, bl, st), "reduce of 8 regions")
    out["stream_reduce_8_regions_gbs"], out["stream_reduce_8_regions_blocks"] = round(gbs, 1), bl
    torch.cuda.synchronize()
    del a, b
    ex = bench_executor_copy(device, iters=iters, nbytes=nbytes)
    out["executor_copy_gbs"] = round(ex["gbs"], 1)
    out["executor_copy_frac_of_stream_copy"] = round(ex["gbs"] / out["stream_copy_gbs"], 4)
    return out


def bench_executor_copy(device, iters=20, nbytes=1 << 30):
    """The executor's own copy path on one contiguous 1 GiB buffer (a one-rank AllToAllv: the
    aligned-copy kernel, 8 KiB tiles): a streaming-copy reference measured with the library's
    code, and the known-size kernel that scales the FETCH_SIZE / WRITE_SIZE counters."""
    import torch

    import paper_2608_00358_amd as H

    n = nbytes // 2
    src = torch.empty(n, dtype=torch.bfloat16, device=device).fill_(1.5)
    dst = torch.empty_like(src)
    with H.Comm(1, device=0) as c:
        call = c.bind_alltoallv([src], [n], [0], [dst], [n], [0])
        for _ in range(3):
            call()
        ms = _time_events(call, iters)
        info = c.last_program()
    torch.cuda.synchronize()
    assert bool(torch.equal(src, dst))
    return {"workload": "executor copy of one contiguous 1 GiB buffer (one-rank AllToAllv)", "bytes_read": nbytes,
            "bytes_written": nbytes, "us": ms * 1e3, "gbs": 2 * nbytes / (ms * 1e-3) / 1e9,
            "tiles": info["num_tiles"], "workers": info["workers"]}


def bench_two_level_c4(device, iters=10, unfused=True):
    """Two-level all-reduce P=64 (8 groups x 8) x 32 MiB bf16 N(0,1)."""
    import torch

    import paper_2608_00358_amd as H
    from workloads import device_normal_bf16

    P, L = 64, 8
    N = 32 * MiB // 2
    send = device_normal_bf16(P, N, seed=0, device=device)
    recv = [torch.empty(N, dtype=torch.bfloat16, device=device) for _ in range(P)]
    algo = 2 * P * N * 2
    out = {"workload": "allreduce two-level P=64 (8x8) 32MiB/rank bf16", "algo_bytes": algo}
    with H.Comm(P, device=0, algo="two_level", group_size=L) as c:
        c.allreduce(send, recv)
        ms = _time_events(lambda: c.allreduce(send, recv), iters)
        info = c.last_program()
        out.update({"us": ms * 1e3, "gbs": algo / (ms * 1e-3) / 1e9, "descs": info["num_descs"],
                    "compile_us": round(info["compile_us"], 1), "launches": info["num_phases"],
                    "schedule_bytes": info["bytes_read"] + info["bytes_written"],
                    "tiles": info["num_tiles"], "workers": info["workers"]})
        if not unfused:
            out["frac"] = out["gbs"] / HBM_PEAK_GBS
            return out
        # the same program as one launch: every reduction writes all 64 ranks itself
        c.set_config(algo="two_level", group_size=L, phases="one")
        c.allreduce(send, recv)
        ms1 = _time_events(lambda: c.allreduce(send, recv), iters)
        out.update({"one_launch_us": ms1 * 1e3, "one_launch_gbs": algo / (ms1 * 1e-3) / 1e9})
        c.set_config(algo="two_level", group_size=L)
        # the same sum in the flat ascending order (one 64-source fold per element): its time,
        # and how far the two-level tree order's results lie from it
        flat = [torch.empty(N, dtype=torch.bfloat16, device=device) for _ in range(P)]
        c.set_config(algo="ring")
        c.allreduce(send, flat)
        ms_flat = _time_events(lambda: c.allreduce(send, flat), iters)
        d = _bf16_ulp_distance(recv[0], flat[0])
        out.update({"flat_ascending_us": ms_flat * 1e3, "flat_ascending_gbs": algo / (ms_flat * 1e-3) / 1e9,
                    "tree_vs_flat_differ": int((d > 0).sum()), "tree_vs_flat_above_1ulp": int((d > 1).sum()),
                    "tree_vs_flat_max_ulp": int(d.max()), "elements": N})
        del flat
        for phases in ("auto", "one"):
            c.set_config(algo="two_level", group_size=L, fuse=0, phases=phases)
            c.allreduce(send, recv)
            ms = _time_events(lambda: c.allreduce(send, recv), iters)
            info = c.last_program()
            key = "unfused" if phases == "auto" else "unfused_one_launch"
            out.update({f"{key}_us": ms * 1e3, f"{key}_gbs": algo / (ms * 1e-3) / 1e9,
                        f"{key}_launches": info["num_phases"],
                        f"{key}_schedule_bytes": info["bytes_read"] + info["bytes_written"]})
    out["frac"] = out["gbs"] / HBM_PEAK_GBS
    del send, recv
    torch.cuda.empty_cache()
    return out


def bench_latency_c5b(device, warmup=100, iters=1000, isolated=200):
    """All-reduce P=8 x 64 KiB fp32, one-shot schedule: back-to-back and isolated latency."""
    import torch

    import paper_2608_00358_amd as H
    from workloads import uniform_f32

    P, N = 8, 1 << 14
    x = uniform_f32(P, N, seed=5)
    send = [torch.from_numpy(x[r].copy()).to(device) for r in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device=device) for _ in range(P)]
    with H.Comm(P, device=0, algo="direct") as c:
        for _ in range(warmup):
            c.allreduce(send, recv)
        ms_marshal = _time_events(lambda: c.allreduce(send, recv), iters)
        call = c.bind_allreduce(send, recv)
        ms = _time_events(call, iters)
        s = torch.cuda.current_stream()
        samples = []
        for _ in range(isolated):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record(s)
            call()
            b.record(s)
            b.synchronize()
            samples.append(a.elapsed_time(b) * 1e3)
        t_host = []
        for _ in range(isolated):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            call()
            torch.cuda.synchronize()
            t_host.append((time.perf_counter() - t0) * 1e6)
        # host cost of re-enqueueing the cached packet (one ctypes call and one launch; the
        # paper keeps this under 10 us, Section V-B)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(200):
            call()
        enqueue_us = (time.perf_counter() - t0) * 1e6 / 200
        torch.cuda.synchronize()
        info = c.last_program()
    # floor: a one-element torch fill launched back to back on the same stream
    tiny = torch.zeros(1, device=device)
    empty_ms = _time_events(lambda: tiny.fill_(1.0), iters)
    return {"workload": "allreduce direct P=8 64KiB/rank fp32", "back_to_back_us": ms * 1e3,
            "back_to_back_with_python_marshalling_us": ms_marshal * 1e3,
            "tiny_torch_kernel_back_to_back_us": empty_ms * 1e3, "inline_launch": info["inline_launch"],
            "isolated_median_us": statistics.median(samples),
            "host_roundtrip_median_us": statistics.median(t_host), "host_enqueue_us": enqueue_us,
            "compile_us": round(info["compile_us"], 1), "workers": info["workers"], "tiles": info["num_tiles"]}


def bench_resident_c5b(device, blocks=0, warmup=200, iters=1000):
    """The same 64 KiB all-reduce handed to the resident executor through the host doorbell:
    host round trip (submit, then poll pinned memory until the packet is reported complete) and
    back-to-back rate (submit `iters` packets, then wait for the last), beside the launched
    kernel's round trip (launch, then synchronise the stream)."""
    import torch

    import paper_2608_00358_amd as H
    from workloads import uniform_f32

    P, N = 8, 1 << 14
    x = uniform_f32(P, N, seed=5)
    send = [torch.from_numpy(x[r].copy()).to(device) for r in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device=device) for _ in range(P)]
    s = torch.cuda.current_stream()
    with H.Comm(P, device=0, algo="direct") as c:
        call = c.bind_allreduce(send, recv)
        for _ in range(warmup):
            call()
        torch.cuda.synchronize()
        launched = []
        for _ in range(iters):
            t0 = time.perf_counter()
            call()
            s.synchronize()
            launched.append((time.perf_counter() - t0) * 1e6)
        with c.resident(blocks=blocks, idle_ms=20000):
            for _ in range(warmup):
                call()
            c.resident_wait(timeout_ms=10000)
            rt = []
            for _ in range(iters):
                t0 = time.perf_counter()
                call()
                c.resident_wait()
                rt.append((time.perf_counter() - t0) * 1e6)
            t0 = time.perf_counter()
            for _ in range(iters):
                call()
            c.resident_wait(timeout_ms=10000)
            b2b = (time.perf_counter() - t0) * 1e6 / iters
            t0 = time.perf_counter()
            for _ in range(iters):
                H.hccl_resident_last_seq(c.handle)     # the cost of one ctypes call, for scale
            ctypes_us = (time.perf_counter() - t0) * 1e6 / iters
    return {"workload": "allreduce direct P=8 64KiB/rank fp32, resident executor",
            "blocks": blocks or 32, "resident_roundtrip_median_us": statistics.median(rt),
            "resident_roundtrip_p99_us": sorted(rt)[int(0.99 * len(rt))],
            "resident_back_to_back_us": b2b,
            "launched_roundtrip_median_us": statistics.median(launched),
            "ctypes_call_us": ctypes_us}


class _HipStream:
    """A HIP stream created through ctypes (CU-masked, or non-blocking), at the default
    priority. Used as a context manager: on exit it is synchronised and destroyed, so that no
    stream of ours is left for the runtime to tear down at process exit."""

    def __init__(self, mask_words=None):
        import torch

        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
        s = ctypes.c_void_p()
        if mask_words is not None:
            self._hip.hipExtStreamCreateWithCUMask.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32,
                                                               ctypes.POINTER(ctypes.c_uint32)]
            arr = (ctypes.c_uint32 * len(mask_words))(*mask_words)
            rc = self._hip.hipExtStreamCreateWithCUMask(ctypes.byref(s), len(mask_words), arr)
            what = "hipExtStreamCreateWithCUMask"
        else:
            self._hip.hipStreamCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32]
            rc = self._hip.hipStreamCreateWithFlags(ctypes.byref(s), 1)   # hipStreamNonBlocking
            what = "hipStreamCreateWithFlags"
        if rc != 0:
            raise RuntimeError(f"{what} failed ({rc})")
        self.handle = s.value
        self.stream = torch.cuda.ExternalStream(self.handle)

    def __enter__(self):
        return self.stream

    def __exit__(self, *exc):
        self.stream.synchronize()
        self._hip.hipStreamDestroy(self.handle)
        self.handle = None
        return False


def _first_cus_mask(n_per_xcd_total):
    """Mask words selecting the first n bits (bit i is a CU of XCD i mod 8)."""
    import torch

    words = (torch.cuda.get_device_properties(0).multi_processor_count + 31) // 32
    bits = [0] * words
    for i in range(n_per_xcd_total):
        bits[i // 32] |= 1 << (i % 32)
    return bits


def bench_overlap_c5a(device, rs_send, rs_recv, n_rs=100, rs_cus=16):
    """Reduce-scatter (c3 shape) on a stream masked to 16 CUs while a bf16 8192^3 GEMM runs on
    a second stream (all CUs, and the 240 complementary CUs)."""
    import torch

    import paper_2608_00358_amd as H

    props = torch.cuda.get_device_properties(0)
    ncu = props.multi_processor_count
    words = (ncu + 31) // 32
    rs_bits = _first_cus_mask(rs_cus)
    rest_bits = [((~rs_bits[w]) & 0xFFFFFFFF) for w in range(words)]
    if ncu % 32:
        rest_bits[-1] &= (1 << (ncu % 32)) - 1
    with _HipStream(rs_bits) as rs_stream, _HipStream(rest_bits) as rest_stream:
        return _overlap_c5a(device, rs_send, rs_recv, n_rs, rs_stream, rest_stream)


def _overlap_c5a(device, rs_send, rs_recv, n_rs, rs_stream, rest_stream):
    import torch

    import paper_2608_00358_amd as H

    gemm_stream = torch.cuda.Stream()
    n = 8192
    g = torch.Generator(device=device).manual_seed(0)
    A = torch.randn(n, n, device=device, dtype=torch.bfloat16, generator=g)
    B = torch.randn(n, n, device=device, dtype=torch.bfloat16, generator=g)
    C = torch.empty(n, n, device=device, dtype=torch.bfloat16)
    flop = 2.0 * n ** 3

    def gemm_time(stream, iters=20):
        with torch.cuda.stream(stream):
            for _ in range(3):
                torch.matmul(A, B, out=C)
            return _time_events(lambda: torch.matmul(A, B, out=C), iters, stream)

    t_all = gemm_time(gemm_stream)
    t_240 = gemm_time(rest_stream)
    P = len(rs_send)
    M = rs_recv[0].numel()
    algo = (P + 1) * P * M * 2
    comm = H.Comm(P, device=0, algo="ring", chunk_bytes=MiB)
    comm.reduce_scatter(rs_send, rs_recv, stream=rs_stream)  # compile and upload outside the timing
    rs_stream.synchronize()
    rs_ms = _time_events(lambda: comm.reduce_scatter(rs_send, rs_recv, stream=rs_stream), 5, rs_stream)
    workers = comm.last_program()["workers"]
    # on a few CUs the bound is what those CUs move, not HBM: the plain 8-region sum on the
    # same masked stream is this case's ceiling
    plain_ms = _plain_reduce_ms(device, rs_stream, P * M * 2, streams=P)
    # overlap: n_rs back-to-back reduce-scatters on the masked stream, GEMMs alongside
    n_gemm = max(5, int(0.9 * n_rs * rs_ms / t_all))
    results = {}
    for label, gstream in (("all_cus", gemm_stream), ("complement_cus", rest_stream)):
        torch.cuda.synchronize()
        ev = {k: torch.cuda.Event(enable_timing=True) for k in ("rs0", "rs1", "g0", "g1")}
        ev["rs0"].record(rs_stream)
        for _ in range(n_rs):
            comm.reduce_scatter(rs_send, rs_recv, stream=rs_stream)
        ev["rs1"].record(rs_stream)
        with torch.cuda.stream(gstream):
            ev["g0"].record(gstream)
            for _ in range(n_gemm):
                torch.matmul(A, B, out=C)
            ev["g1"].record(gstream)
        torch.cuda.synchronize()
        g_ms = ev["g0"].elapsed_time(ev["g1"]) / n_gemm
        r_ms = ev["rs0"].elapsed_time(ev["rs1"]) / n_rs
        base = t_all if label == "all_cus" else t_240
        results[label] = {"gemm_ms": g_ms, "gemm_tflops": flop / (g_ms * 1e-3) / 1e12,
                          "gemm_slowdown_pct": (g_ms / base - 1.0) * 100.0,
                          "rs_ms": r_ms, "rs_gbs": algo / (r_ms * 1e-3) / 1e9}
    if comm.async_error() != 0:
        raise RuntimeError(H.hccl_get_last_error())
    comm.close()
    return {"workload": "reduce_scatter P=8 256MiB/rank bf16 on 16 CUs || bf16 8192^3 GEMM",
            "gemm_alone_all_cus_ms": t_all, "gemm_alone_all_cus_tflops": flop / (t_all * 1e-3) / 1e12,
            "gemm_alone_240_cus_ms": t_240, "rs_alone_16cu_ms": rs_ms,
            "rs_alone_16cu_gbs": algo / (rs_ms * 1e-3) / 1e9, "rs_workers": workers,
            "plain_reduce_16cu_ms": plain_ms, "plain_reduce_16cu_gbs": algo / (plain_ms * 1e-3) / 1e9,
            "rs_alone_16cu_frac_of_plain_reduce": plain_ms / rs_ms,
            "n_rs": n_rs, "n_gemm": n_gemm, "overlap": results}


# ------------------------------------------------------------------ AllToAllvDynamic
def bench_dynamic_alltoallv(device, w, iters=20, plan_only=True):
    """The headline exchange with its count matrix in device memory (hccl_alltoallv_dynamic,
    rows and ids grouped, one launch): time per launch against the host-layout AllToAllv, and
    (plan_only) the fixed cost of the on-device plan (an exchange whose counts are all zero)."""
    import numpy as np
    import torch

    import paper_2608_00358_amd as H

    P, R, D = w["P"], w["R"], w["D"]
    counts = w["counts"]
    cap = int(counts.sum(axis=0).max())
    send_rows = w["send_rows"]
    send_ids = [torch.from_numpy(w["id_vals"][s].copy()).to(device) for s in range(P)]
    recv_rows = [torch.empty(cap * D, dtype=torch.bfloat16, device=device) for _ in range(P)]
    recv_ids = [torch.empty(cap, dtype=torch.int32, device=device) for _ in range(P)]
    d_counts = torch.from_numpy(counts.reshape(-1).astype(np.int64)).to(device)
    d_zero = torch.zeros_like(d_counts)
    algo = 2 * int(counts.sum()) * (D * 2 + 4)
    out = {"workload": "alltoallv_dynamic P=8, 2^18 rows/rank of 128 bf16 + int32 ids, Zipf(1.1), counts in "
                       "device memory, rows and ids grouped (one launch)", "algo_bytes": algo}
    with H.Comm(P, device=0) as c:
        def step(dc):
            H.hccl_group_start(c.handle)
            calls[dc][0]()
            calls[dc][1]()
            H.hccl_group_end(c.handle)

        calls = {}
        for key, dc in (("full", d_counts), ("zero", d_zero)):
            calls[key] = (c.bind_alltoallv_dynamic(send_rows, dc, recv_rows, D),
                          c.bind_alltoallv_dynamic(send_ids, dc, recv_ids, 1))
        for _ in range(3):
            step("full")
        ms = _time_events(lambda: step("full"), iters)
        info = c.last_program()
        ms_zero = _time_events(lambda: step("zero"), iters) if plan_only else None
        if c.async_error() != 0:
            raise RuntimeError(H.hccl_get_last_error())
    out.update({"us": ms * 1e3, "gbs": algo / (ms * 1e-3) / 1e9, "frac": algo / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "tiles": info["num_tiles"], "workers": info["workers"]})
    if ms_zero is not None:
        out["plan_only_us"] = ms_zero * 1e3
    return out


def bench_moe_dispatch(device, iters=60, warmup=10):
    """Routing on the GPU followed by the dispatch exchange, every iteration a new routing:
    (a) device-resident: routing, then hccl_alltoallv_dynamic on the same stream, no host step;
    (b) eager: routing, copy the counts to the host, build the layout, hccl_alltoallv (a new
    program whenever the counts change). Wall time per iteration, synchronised at its end."""
    import numpy as np
    import torch

    import paper_2608_00358_amd as H

    P, T, D = 8, 256, 4096      # 256 tokens of 4096 bf16 per rank: 2 MiB per rank
    g = torch.Generator(device=device)
    g.manual_seed(7)
    tokens = torch.randn(P, T, D, generator=g, device=device).to(torch.bfloat16)
    send_all = torch.empty(P, T * D, dtype=torch.bfloat16, device=device)
    send = [send_all[s] for s in range(P)]
    cap = P * T
    recv = [torch.empty(cap * D, dtype=torch.bfloat16, device=device) for _ in range(P)]
    d_counts = torch.empty(P * P, dtype=torch.int64, device=device)
    rank_base = (torch.arange(P, device=device) * P).view(P, 1)

    def route():
        # skewed destinations, per-(source, destination) counts, tokens sorted by destination
        dest = (torch.rand(P, T, generator=g, device=device) ** 2 * P).long().clamp_(max=P - 1)
        d_counts.copy_(torch.bincount((dest + rank_base).view(-1), minlength=P * P))
        order = torch.argsort(dest, dim=1, stable=True)
        torch.take_along_dim(tokens, order.unsqueeze(-1), dim=1, out=send_all.view(P, T, D))

    def timed(fn):
        samples = []
        for i in range(warmup + iters):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            if i >= warmup:
                samples.append((time.perf_counter() - t0) * 1e6)
        return statistics.median(samples)

    with H.Comm(P, device=0) as c:
        dyn = c.bind_alltoallv_dynamic(send, d_counts, recv, D)

        def eager():
            route()
            counts = d_counts.cpu().numpy().reshape(P, P)
            sd = np.zeros((P, P), np.int64)
            rd = np.zeros((P, P), np.int64)
            sd[:, 1:] = np.cumsum(counts, axis=1)[:, :-1] * D
            rd[:, 1:] = np.cumsum(counts.T, axis=1)[:, :-1] * D
            H.hccl_alltoallv(c.handle, send, counts * D, sd, recv, counts.T * D, rd, "bf16")

        t_route = timed(route)
        t_dyn = timed(lambda: (route(), dyn()))
        t_eager = timed(eager)
        if c.async_error() != 0:
            raise RuntimeError(H.hccl_get_last_error())
    return {"workload": "MoE dispatch P=8, 256 tokens x 4096 bf16 per rank, skewed routing on the GPU each "
                        "iteration", "route_only_us": t_route, "device_resident_us": t_dyn, "eager_host_layout_us": t_eager,
            "exchange_exposed_device_resident_us": t_dyn - t_route,
            "exchange_exposed_eager_us": t_eager - t_route}


def bench_triggered_dispatch(device, iters=60, warmup=10, per_xcd=16, done_word=True):
    """Routing followed by the dispatch exchange, the compute side on its own stream:
    (a) eager: counts to the host, layout, hccl_alltoallv on the compute stream;
    (b) device-resident: hccl_alltoallv_dynamic on the compute stream right after routing;
    (c) device-resident and device-triggered: the dynamic exchange is enqueued first on a stream
        masked to `per_xcd` CUs per XCD and waits on a device word; routing ends by writing it.
    Wall time per iteration (synchronised at its end), and the exposed exchange time from the
    end of routing to the end of the exchange (HIP events)."""
    import numpy as np
    import torch

    import paper_2608_00358_amd as H

    P, T, D = 8, 256, 4096
    g = torch.Generator(device=device)
    g.manual_seed(11)
    tokens = torch.randn(P, T, D, generator=g, device=device).to(torch.bfloat16)
    send_all = torch.empty(P, T * D, dtype=torch.bfloat16, device=device)
    send = [send_all[s] for s in range(P)]
    cap = P * T
    recv = [torch.empty(cap * D, dtype=torch.bfloat16, device=device) for _ in range(P)]
    d_counts = torch.empty(P * P, dtype=torch.int64, device=device)
    flag = torch.zeros(1, dtype=torch.int64, device=device)
    done = torch.zeros(1, dtype=torch.int64, device=device)
    rank_base = (torch.arange(P, device=device) * P).view(P, 1)
    with _HipStream() as cs, _HipStream(_first_cus_mask(8 * per_xcd)) as ms:
        return _triggered_dispatch(device, iters, warmup, per_xcd, done_word, P, T, D, g, tokens, send_all, send,
                                   recv, d_counts, flag, done, rank_base, cs, ms)


def _triggered_dispatch(device, iters, warmup, per_xcd, done_word, P, T, D, g, tokens, send_all, send, recv,
                        d_counts, flag, done, rank_base, cs, ms):
    import numpy as np
    import torch

    import paper_2608_00358_amd as H

    def route():
        dest = (torch.rand(P, T, generator=g, device=device) ** 2 * P).long().clamp_(max=P - 1)
        d_counts.copy_(torch.bincount((dest + rank_base).view(-1), minlength=P * P))
        order = torch.argsort(dest, dim=1, stable=True)
        torch.take_along_dim(tokens, order.unsqueeze(-1), dim=1, out=send_all.view(P, T, D))

    out = {"workload": "MoE dispatch P=8, 256 tokens x 4096 bf16 per rank, GPU routing on a compute stream, "
                       f"triggered exchange on {8 * per_xcd} CUs"}
    with H.Comm(P, device=0) as c:
        dyn_c = c.bind_alltoallv_dynamic(send, d_counts, recv, D, stream=cs)

        def eager():
            route()
            counts = d_counts.cpu().numpy().reshape(P, P)   # waits for the compute stream
            sd = np.zeros((P, P), np.int64)
            rd = np.zeros((P, P), np.int64)
            sd[:, 1:] = np.cumsum(counts, axis=1)[:, :-1] * D
            rd[:, 1:] = np.cumsum(counts.T, axis=1)[:, :-1] * D
            H.hccl_alltoallv(c.handle, send, counts * D, sd, recv, counts.T * D, rd, "bf16", stream=cs)

        def timed(body, exposed, pre=None):
            wall, exp = [], []
            for i in range(warmup + iters):
                if pre:
                    pre(i)   # enqueued ahead of the compute work, outside the timed region
                time.sleep(0.0002)
                t0 = time.perf_counter()
                e = body(i)
                torch.cuda.synchronize()
                if i >= warmup:
                    wall.append((time.perf_counter() - t0) * 1e6)
                    if exposed:
                        exp.append(e[0].elapsed_time(e[1]) * 1e3)
            return statistics.median(wall), (statistics.median(exp) if exp else None)

        def run_eager(i):
            with torch.cuda.stream(cs):
                eager()

        def run_resident(i):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            with torch.cuda.stream(cs):
                route()
                a.record(cs)
                dyn_c()
                b.record(cs)
            return a, b

        seq = [0]
        dyn_m = c.bind_alltoallv_dynamic(send, d_counts, recv, D, stream=ms)

        def prelaunch(i):
            torch.cuda.synchronize()
            seq[0] += 1
            v = seq[0]
            H.hccl_set_trigger(c.handle, (flag, "ge", v), (done, v) if done_word else None)
            dyn_m()   # the exchange is resident and waiting before routing starts

        def run_triggered(i):
            v = seq[0]
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            with torch.cuda.stream(cs):
                route()
                flag.fill_(v)
                a.record(cs)
            b.record(ms)
            return a, b

        out["eager_wall_us"], _ = timed(run_eager, False)
        out["resident_wall_us"], out["resident_exposed_us"] = timed(run_resident, True)
        out["triggered_wall_us"], out["triggered_exposed_us"] = timed(run_triggered, True, prelaunch)
        if c.async_error() != 0:
            raise RuntimeError(H.hccl_get_last_error())
        if done_word and int(done.item()) != seq[0]:
            raise RuntimeError("completion word not written")
    route_only = []
    for i in range(warmup + iters):
        torch.cuda.synchronize()
        time.sleep(0.0002)
        t0 = time.perf_counter()
        with torch.cuda.stream(cs):
            route()
        torch.cuda.synchronize()
        if i >= warmup:
            route_only.append((time.perf_counter() - t0) * 1e6)
    out["route_only_wall_us"] = statistics.median(route_only)
    torch.cuda.synchronize()
    return out


# ---------------------------------------------------------------------- CPU baseline
def _cpu_description():
    """CPU model and topology of the host, from lscpu (falls back to /proc/cpuinfo)."""
    import subprocess

    keys = ("Model name", "Vendor ID", "CPU family", "Model", "Thread(s) per core", "Core(s) per socket",
            "Socket(s)", "CPU(s)", "On-line CPU(s) list", "CPU max MHz", "L3 cache")
    out = {}
    try:
        text = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in text.splitlines():
            k, _, v = line.partition(":")
            if k.strip() in keys:
                out[k.strip()] = v.strip()
    except (OSError, subprocess.SubprocessError):
        pass
    if "Model name" not in out:
        try:
            for line in open("/proc/cpuinfo"):
                if line.startswith("model name"):
                    out["Model name"] = line.split(":", 1)[1].strip()
                    break
        except OSError:
            pass
    try:
        out["affinity_cpus"] = len(os.sched_getaffinity(0))
    except OSError:
        pass
    return out


def _pair_groups(sendcounts, n):
    """(source, destination) pairs split into n groups of about equal element counts."""
    P = sendcounts.shape[0]
    pairs = sorted(((int(sendcounts[s, d]), s, d) for s in range(P) for d in range(P)), reverse=True)
    groups, load = [[] for _ in range(n)], [0] * n
    for c, s, d in pairs:
        k = load.index(min(load))
        groups[k].append((s, d))
        load[k] += c
    return [g for g in groups if g]


def _masked(lay, pairs):
    """The layout with every count outside `pairs` set to zero (send [s, d], receive [d, s])."""
    import numpy as np

    sc = np.zeros_like(lay["sendcounts"])
    for s, d in pairs:
        sc[s, d] = lay["sendcounts"][s, d]
    return sc, sc.T.copy()


def cpu_baseline(w, budget_s=10.0, par_budget_s=5.0):
    """The oracle's AllToAllv of the timed step (embedding rows and int32 ids, the same inputs)
    on the host cores: single-threaded, then chunk-parallel (host threads each run the
    unchanged oracle on their own (source, destination) pairs; the oracle releases the GIL).
    The oracle's result is compared element by element with what the GPU left in the receive
    buffers after its last timed step."""
    import numpy as np
    import torch
    from concurrent.futures import ThreadPoolExecutor

    import oracle

    P = w["P"]
    rows, ids = w["rows"], w["ids"]
    send_r = [t.view(torch.int16).cpu().numpy().view(np.uint16) for t in w["send_rows"]]
    send_i = [np.ascontiguousarray(w["id_vals"][s]) for s in range(P)]
    got_r = [t.view(torch.int16).cpu().numpy().view(np.uint16) for t in w["recv_rows"]]
    got_i = [t.cpu().numpy() for t in w["recv_ids"]]
    oracle.build(force=False)
    out_r = [np.zeros(int(rows["recv_len"][d]), np.uint16) for d in range(P)]
    out_i = [np.zeros(int(ids["recv_len"][d]), np.int32) for d in range(P)]

    def step():
        oracle.alltoallv(send_r, rows["sendcounts"], rows["sdispls"], out_r, rows["recvcounts"], rows["rdispls"])
        oracle.alltoallv(send_i, ids["sendcounts"], ids["sdispls"], out_i, ids["recvcounts"], ids["rdispls"])

    reps, t = 0, 0.0
    while t < budget_s and reps < 100:
        t0 = time.perf_counter()
        step()
        t += time.perf_counter() - t0
        reps += 1
    verified = all(np.array_equal(got_r[d], out_r[d]) and np.array_equal(got_i[d], out_i[d]) for d in range(P))
    mism = [d for d in range(P) if not (np.array_equal(got_r[d], out_r[d]) and np.array_equal(got_i[d], out_i[d]))]

    nthreads = max(1, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1))
    groups = _pair_groups(rows["sendcounts"], nthreads)
    masks = [(_masked(rows, g), _masked(ids, g)) for g in groups]
    par_r = [np.zeros_like(o) for o in out_r]
    par_i = [np.zeros_like(o) for o in out_i]

    def part(k):
        (rs, rr), (is_, ir) = masks[k]
        oracle.alltoallv(send_r, rs, rows["sdispls"], par_r, rr, rows["rdispls"])
        oracle.alltoallv(send_i, is_, ids["sdispls"], par_i, ir, ids["rdispls"])

    preps, pt = 0, 0.0
    with ThreadPoolExecutor(max_workers=len(groups)) as pool:
        while pt < par_budget_s and preps < 200:
            t0 = time.perf_counter()
            list(pool.map(part, range(len(groups))))
            pt += time.perf_counter() - t0
            preps += 1
    par_same = all(np.array_equal(par_r[d], out_r[d]) and np.array_equal(par_i[d], out_i[d]) for d in range(P))

    algo = 2 * (int(rows["sendcounts"].sum()) * 2 + int(ids["sendcounts"].sum()) * 4)
    return {"value": algo * reps / t / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"the timed step's AllToAllv (8 ranks x 64 MiB bf16 rows + 1 MiB int32 ids, the same "
                      f"inputs), {reps} full repetitions in {t:.1f}s, single-threaded C oracle",
            "verified": bool(verified), "verified_what": "every element of the GPU's receive buffers after the "
                                                           "last timed step equals the oracle's result",
            "mismatched_destinations": mism,
            "parallel": {"value": algo * preps / pt / 1e9, "unit": "GB/s", "cores": len(groups),
                         "sample": f"{preps} repetitions in {pt:.1f}s, {len(groups)} host threads, each running "
                                   f"the oracle on its share of the 64 (source, destination) pairs",
                         "same_result": bool(par_same)},
            "cpu": _cpu_description(), "host_threads_available": os.cpu_count()}


# ------------------------------------------------------------------------ roofline
def traffic_record(kernel: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were taken on
    the current executor source (otherwise null)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except ValueError:
        return None
    src = os.path.join(ROOT, "paper_2608_00358_amd", "csrc", "executor.hip")
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    entry = rec.get(kernel)
    if not entry or entry.get("executor_sha256_16") != digest:
        return None
    return entry.get("bytes_per_launch")


def _only_c3(device):
    res, send, recv = bench_reduce_scatter_c3(device)
    del send, recv
    return res


def _only_c5a(device):
    """The overlap measurement alone: the c3 inputs, every reduce-scatter on the masked stream."""
    import torch

    from workloads import device_normal_bf16

    P = 8
    M = (256 * MiB // 2) // P
    send = device_normal_bf16(P, P * M, std=0.02, seed=0, device=device)
    recv = [torch.empty(M, dtype=torch.bfloat16, device=device) for _ in range(P)]
    res = bench_overlap_c5a(device, send, recv)
    del send, recv
    return res


# single measurements for profiling runs (bench.py --only NAME)
ONLY = {
    "copy": bench_executor_copy,
    "c1": bench_allreduce_ring_c1,
    "c3": _only_c3,
    "c4": lambda d: bench_two_level_c4(d, unfused=False),
    "c4_both": bench_two_level_c4,
    "c5a": _only_c5a,
    "c5b": bench_latency_c5b,
    "orders": bench_forwarded_partials,
    "ceiling": bench_copy_ceiling,
}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--headline-only", action="store_true", help="only the timed AllToAllv steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-overlap", action="store_true")
    ap.add_argument("--latency-only", action="store_true", help="only the 64 KiB all-reduce latency test")
    ap.add_argument("--dynamic-only", action="store_true",
                    help="only the AllToAllvDynamic measurements (headline exchange, MoE dispatch)")
    ap.add_argument("--dynamic-exchange-only", action="store_true",
                    help="only the AllToAllvDynamic form of the headline exchange")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run torch's device copy of 1 GiB")
    ap.add_argument("--only", choices=sorted(ONLY), help="run one secondary measurement and print it")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the P ranks are buffers in one MI355X's HBM; "
              "the library has no multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    import paper_2608_00358_amd as H

    H.load()
    device = "cuda:0"
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=device)
        a.fill_(1)
        b = torch.empty_like(a)
        ms = _time_events(lambda: b.copy_(a), 5)
        print(json.dumps({"calibration": "torch copy_ 1 GiB", "bytes_read": 1 << 30, "bytes_written": 1 << 30,
                          "us": ms * 1e3}), flush=True)
        return

    if args.only:
        print(json.dumps({args.only: ONLY[args.only](device)}), flush=True)
        return

    if args.latency_only:
        print(json.dumps(bench_latency_c5b(device)), flush=True)
        for blocks in (1, 2, 4, 8, 32):
            print(json.dumps(bench_resident_c5b(device, blocks=blocks)), flush=True)
        return

    if args.dynamic_exchange_only:
        w = alltoallv_workload(device)
        print(json.dumps({"alltoallv_dynamic_rows_ids_p8": bench_dynamic_alltoallv(device, w, plan_only=False)}),
              flush=True)
        return

    if args.dynamic_only:
        w = alltoallv_workload(device)
        print(json.dumps({"alltoallv_dynamic_rows_ids_p8": bench_dynamic_alltoallv(device, w),
                          "moe_dispatch_p8": bench_moe_dispatch(device),
                          "moe_dispatch_triggered_p8": bench_triggered_dispatch(device)}), flush=True)
        return

    head, w = run_headline(args, device)
    _log(f"alltoallv step {head['ms_per_step']:.3f} ms, {head['value']:.1f} GB/s; "
         f"launch {head['launch_ms'] * 1e3:.1f} us")
    achieved = head["algo_bytes_step"] / (head["launch_ms"] * 1e-3) / 1e9
    traffic = traffic_record("alltoallv_rows_ids_p8_zipf_group")
    line = {
        "metric": "effective HBM GB/s per collective (% of MI355X HBM peak); small-msg latency us",
        "value": round(head["value"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(head["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "alltoallv P=8 virtual ranks, 2^18 rows/rank of 128 bf16 (64 MiB/rank), "
                               "Zipf(1.1) destination split, int32 row ids alongside; both payloads in one "
                               "group (one work packet, one executor launch)",
                   "ranks": 8, "rows_per_rank": 1 << 18, "row_elems": 128,
                   "recv_imbalance_max_over_mean": round(head["recv_imbalance"], 3),
                   "descs": head["program"]["num_descs"], "tiles": head["program"]["num_tiles"],
                   "workers": head["program"]["workers"],
                   "step_tiles_elems": [head["program"]["step_tile_min"], head["program"]["step_tile_max"]],
                   "compile_us": round(head["program"]["compile_us"], 1),
                   "host_enqueue_us_per_step": round(head["host_enqueue_us"], 2)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "kernel": "hccl_executor<12> (copy-only executor; the grouped rows + ids launch)",
                     "algo_bytes_per_launch": head["algo_bytes_step"],
                     "avg_launch_us": round(head["launch_ms"] * 1e3, 2)},
    }
    if head["separate_calls"]:
        line["config"]["separate_calls"] = {k: round(v, 2) for k, v in head["separate_calls"].items()}
    if not args.headline_only:
        _log("copy ceiling")
        ceil = _extra("ceiling", lambda: bench_copy_ceiling(device))
        line["copy_ceiling"] = ceil
        if "stream_copy_gbs" in ceil:
            line["roofline"]["frac_of_stream_copy"] = round(achieved / ceil["stream_copy_gbs"], 4)
    if not args.headline_only:
        extras = {}
        _log("c1 ring all-reduce")
        extras["allreduce_ring_p4_fp32"] = _extra("c1", lambda: bench_allreduce_ring_c1(device))
        _log("c3 ring reduce-scatter")
        c3, rs_send, rs_recv = bench_reduce_scatter_c3(device)
        extras["reduce_scatter_ring_p8_bf16"] = c3
        if not args.headline_only and "stream_reduce_8_regions_gbs" in line.get("copy_ceiling", {}):
            c3["frac_of_stream_reduce"] = round(c3["gbs"] / line["copy_ceiling"]["stream_reduce_8_regions_gbs"], 4)
        _log(f"c3 {c3['gbs']:.1f} GB/s")
        if not args.no_overlap:
            _log("c5a overlap")
            extras["overlap_rs16cu_gemm"] = _extra("c5a overlap", lambda: bench_overlap_c5a(device, rs_send, rs_recv))
        del rs_send, rs_recv
        torch.cuda.empty_cache()
        _log("forwarded-partial schedules and fold orders")
        extras["forwarded_partial_schedules_rs_p8_bf16"] = _extra("orders", lambda: bench_forwarded_partials(device))
        _log("c4 two-level all-reduce")
        extras["allreduce_two_level_p64_bf16"] = _extra("c4", lambda: bench_two_level_c4(device))
        _log("c5b latency")
        extras["latency_allreduce_p8_64KiB_fp32"] = _extra("c5b latency", lambda: bench_latency_c5b(device))
        _log("c5b latency through the resident executor")
        extras["resident_allreduce_p8_64KiB_fp32"] = _extra("resident", lambda: bench_resident_c5b(device))
        _log("alltoallv_dynamic")
        extras["alltoallv_dynamic_rows_ids_p8"] = _extra("dynamic", lambda: bench_dynamic_alltoallv(device, w))
        _log("moe dispatch: device-resident vs eager")
        extras["moe_dispatch_p8"] = _extra("moe", lambda: bench_moe_dispatch(device))
        _log("moe dispatch: device-triggered")
        extras["moe_dispatch_triggered_p8"] = _extra("moe triggered", lambda: bench_triggered_dispatch(device))
        line["collectives"] = extras
    if not args.no_cpu_baseline:
        _log("cpu baseline")
        line["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(line), flush=True)
    if not args.no_cpu_baseline and not line["cpu_baseline"]["verified"]:
        _log("the GPU's receive buffers differ from the oracle's result: the measured step is wrong")
        sys.exit(3)


if __name__ == "__main__":
    main()
