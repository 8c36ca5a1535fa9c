"""Seeded random collectives on the GPU against the oracle, bit for bit.

Case k draws, from seed 1000 + k, a collective, a rank count, an element type, a reduction, a
schedule and its fold order, a phase mode, fusion on or off, chunk and tile sizes, a cap on
the executor's wavefronts and a ragged size. It runs through the C ABI and every output
element, and the guard bands around every output, are compared with the oracle run in the
same fold order (ascending, rotated ring, recursive halving or two-level groups).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import GUARD, Guarded, first_mismatch, same_bits, to_device
from test_gpu_orders import lib_shard
from test_gpu_parity import inputs
from workloads import alltoallv_layout, zipf_counts

pytestmark = pytest.mark.gpu

CASES = 96


def _pow2(P):
    return P >= 2 and P & (P - 1) == 0


def draw(k):
    """Case k: (collective, P, dtype, op, size, library config, oracle order, group)."""
    rng = np.random.default_rng(1000 + k)
    coll = str(rng.choice(["allreduce", "reduce_scatter", "allgather", "alltoallv"], p=[0.4, 0.25, 0.15, 0.2]))
    P = int(rng.choice([1, 2, 3, 4, 5, 8, 12, 16]))
    dt = str(rng.choice(["bf16", "fp16", "fp32", "int32"]))
    cfg = dict(chunk_bytes=int(rng.choice([2048, 8192, 65536, 1 << 20])),
               tile_bytes=int(rng.choice([0, 4096, 16384])),
               max_workers=int(rng.choice([0, 0, 4, 96])),
               phases=str(rng.choice(["auto", "one", "levels"])),
               fuse=int(rng.choice([0, 1])))
    op, order, group = "sum", "ascending", 0
    if coll in ("allreduce", "reduce_scatter"):
        if rng.random() < 0.2:
            op = str(rng.choice(["max", "min"]))
        schedules = [("direct", "ascending"), ("ring", "ascending"), ("ring", "ring")]
        if _pow2(P):
            schedules.append(("rhd", "halving"))
        groups = [L for L in range(2, P) if P % L == 0]
        if coll == "allreduce" and groups:
            schedules += [("two_level", "two_level")] * 2
        algo, order = schedules[int(rng.integers(len(schedules)))]
        cfg["algo"] = algo
        if order != "two_level":
            cfg["order"] = order
        else:
            group = int(rng.choice(groups))
            cfg["group_size"] = group
        size = int(rng.integers(1, 50001)) if coll == "allreduce" else int(rng.integers(1, 6001))
    elif coll == "allgather":
        cfg["algo"] = str(rng.choice(["direct", "ring"] + (["rhd"] if _pow2(P) else [])))
        size = int(rng.integers(1, 9001))
    else:
        cfg.pop("phases")
        cfg["fuse"] = 1
        size = int(rng.integers(1, 3001))  # rows sent per rank
    return coll, P, dt, op, size, cfg, order, group


def _want_reduction(coll, x, dt, op, order, group, N, P):
    if coll == "allreduce":
        if order == "two_level":
            return oracle.allreduce(x, dt, op=op, group=group)
        return oracle.allreduce_ordered(x, dt, order=order, op=op, shard=lib_shard(N, P) if order == "ring" else 0)
    return oracle.reduce_scatter_ordered(x, dt, order=order, op=op)


@pytest.mark.parametrize("k", range(CASES))
def test_random_collective_matches_oracle(k):
    coll, P, dt, op, size, cfg, order, group = draw(k)
    print(f"case {k}: {coll} P={P} dt={dt} op={op} size={size} cfg={cfg} order={order} group={group}", flush=True)
    with H.Comm(P, device=0, **cfg) as c:
        if coll in ("allreduce", "reduce_scatter"):
            n_in = size if coll == "allreduce" else P * size
            x = inputs(P, n_in, dt, seed=k)
            send = [to_device(x[r], dt) for r in range(P)]
            outs = [Guarded(size, dt) for _ in range(P)]
            if coll == "allreduce":
                H.hccl_allreduce(c.handle, send, [o.view for o in outs], size, dt, op)
            else:
                H.hccl_reduce_scatter(c.handle, send, [o.view for o in outs], size, dt, op)
            want = _want_reduction(coll, x, dt, op, order, group, size, P)
        elif coll == "allgather":
            x = inputs(P, size, dt, seed=k)
            send = [to_device(x[r], dt) for r in range(P)]
            outs = [Guarded(P * size, dt) for _ in range(P)]
            H.hccl_allgather(c.handle, send, [o.view for o in outs], size, dt)
            want = oracle.allgather(x)
        else:
            epr = int(np.random.default_rng(k).choice([1, 3, 128]))
            lay = alltoallv_layout(zipf_counts(P, size, 1.1, seed=k), epr)
            x = [inputs(1, max(1, int(lay["send_len"][s])), dt, seed=k * 31 + s)[0][:int(lay["send_len"][s])]
                 for s in range(P)]
            send = [to_device(np.ascontiguousarray(x[s]), dt) for s in range(P)]
            outs = [Guarded(max(1, int(lay["recv_len"][d])), dt) for d in range(P)]
            H.hccl_alltoallv(c.handle, send, lay["sendcounts"], lay["sdispls"], [o.view for o in outs],
                             lay["recvcounts"], lay["rdispls"], dt)
            want = [o.host_init[GUARD:GUARD + o.n].copy() for o in outs]
            oracle.alltoallv([np.ascontiguousarray(a) for a in x], lay["sendcounts"], lay["sdispls"], want,
                             lay["recvcounts"], lay["rdispls"])
        torch.cuda.synchronize()
        assert c.async_error() == 0
    for r in range(P):
        got = outs[r].result()
        if coll == "allgather" or coll == "alltoallv":
            assert np.array_equal(got.view(np.uint8), want[r].view(np.uint8)), f"case {k} rank {r}"
        else:
            assert same_bits(got, want[r], dt), f"case {k} rank {r}: {first_mismatch(got, want[r])}"
        assert outs[r].guards_intact(), f"case {k} rank {r}: guard band overwritten"
