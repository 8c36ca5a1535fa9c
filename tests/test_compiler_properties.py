"""Property tests of the host compiler: every collective the API accepts compiles into a program
that the validator proves well formed (dependency order, operand bounds, no unordered
conflicting accesses, scratch read after write, exact output coverage).

Host-only communicators compile and validate without touching memory, so the search covers
schedules, orders, fusion, phase modes, chunk and tile sizes, groups and dynamic exchanges on the CPU.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import paper_2608_00358_amd as H
from program_interpreter import Program

ES = {"bf16": 2, "fp16": 2, "fp32": 4, "int32": 4}
SETTINGS = settings(max_examples=120, deadline=None, suppress_health_check=[HealthCheck.too_slow])


def fake_bufs(P, base):
    return [base + i * (1 << 36) for i in range(P)]


@st.composite
def reduction_case(draw):
    coll = draw(st.sampled_from(["allreduce", "reduce_scatter", "allgather"]))
    order = draw(st.sampled_from(["ascending", "ring", "halving"]))
    if order == "halving":
        P = draw(st.sampled_from([1, 2, 4, 8, 16, 32]))
        algo = draw(st.sampled_from(["direct", "rhd", "auto"]))
    else:
        P = draw(st.sampled_from([draw(st.integers(1, 12)), 16, 20, 32]))
        algos = ["direct", "ring", "auto"]
        if coll == "allreduce" and order == "ascending":
            algos.append("two_level")
        algo = draw(st.sampled_from(algos))
    if coll == "allgather":
        order = "ascending" if algo != "rhd" else order
    group = 0
    if algo == "two_level":
        divisors = [L for L in range(1, P + 1) if P % L == 0]
        group = draw(st.sampled_from(divisors))
    return dict(coll=coll, P=P, algo=algo, order=order, group=group,
                dt=draw(st.sampled_from(["bf16", "fp16", "fp32", "int32"])),
                op=draw(st.sampled_from(["sum", "max", "min"])),
                count=draw(st.integers(0, 70000)),
                fuse=draw(st.integers(0, 1)),
                requant=draw(st.integers(0, 1)),
                chunk=draw(st.sampled_from([0, 512, 4096, 65536])),
                tile=draw(st.sampled_from([0, 1024, 8192])),
                phases=draw(st.sampled_from(["auto", "one", "levels"])))


@SETTINGS
@given(reduction_case())
def test_every_accepted_reduction_validates(case):
    P = case["P"]
    cfg = dict(algo=case["algo"], order=case["order"], group_size=case["group"], fuse=case["fuse"],
               requantize=case["requant"], chunk_bytes=case["chunk"], tile_bytes=case["tile"], validate=1,
               phases=case["phases"])
    if case["algo"] == "rhd" and case["coll"] != "allgather":
        cfg["order"] = "halving"
    with H.Comm(P, device=H.NO_DEVICE, **cfg) as c:
        s, r = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
        try:
            if case["coll"] == "allreduce":
                H.hccl_allreduce(c.handle, s, r, case["count"], case["dt"], case["op"])
            elif case["coll"] == "reduce_scatter":
                if case["algo"] == "two_level":
                    return
                H.hccl_reduce_scatter(c.handle, s, r, case["count"] // max(P, 1), case["dt"], case["op"])
            else:
                if case["algo"] == "two_level":
                    return
                H.hccl_allgather(c.handle, s, r, case["count"] // max(P, 1), case["dt"])
        except H.HcclError as e:
            # only unsupported combinations may be refused, never with a validation failure
            assert e.code == 2, str(e)
            return
        info = c.last_program()
        assert info["num_descs"] >= 0
        # a launch per level waits for nothing on the device; one launch keeps every wait
        if case["phases"] == "levels" or (case["phases"] == "auto" and info["num_phases"] > 1):
            assert info["num_deps"] == 0
        if case["phases"] == "one":
            assert info["num_phases"] == 1
        check_tile_layout(Program(H.hccl_comm_program_image(c.handle)))


def check_tile_layout(prog):
    """Inside each phase the descriptors own consecutive runs of tiles, in descriptor order, each
    run starting at the descriptor's tile0 and as long as its ntiles (so in a phase whose
    descriptors all have K tiles, tile t belongs to descriptor d0 + (t - t0) // K)."""
    for q in range(len(prog.phase_tile) - 1):
        t0, t1 = int(prog.phase_tile[q]), int(prog.phase_tile[q + 1])
        if t0 == t1:
            continue
        owners = prog.tile_desc[t0:t1].astype(np.int64)
        d0, d1 = int(owners[0]), int(owners[-1]) + 1
        assert (np.diff(owners) >= 0).all() and (np.diff(owners) <= 1).all()
        for d in range(d0, d1):
            assert int(prog.descs[d]["tile0"]) == t0 + int(np.searchsorted(owners, d))
            assert int(prog.descs[d]["ntiles"]) == int((owners == d).sum())
        K = prog.descs[d0:d1]["ntiles"]
        if (K == K[0]).all():
            assert np.array_equal(owners, d0 + (np.arange(t1 - t0) // int(K[0])))


@st.composite
def alltoallv_case(draw):
    P = draw(st.integers(1, 10))
    counts = np.array(draw(st.lists(st.integers(0, 3000), min_size=P * P, max_size=P * P))).reshape(P, P)
    gap = draw(st.integers(0, 37))
    return P, counts, gap, draw(st.sampled_from(["bf16", "int32"])), draw(st.sampled_from([0, 1024, 65536]))


@SETTINGS
@given(alltoallv_case())
def test_every_alltoallv_layout_validates(case):
    P, counts, gap, dt, chunk = case
    sd = np.zeros((P, P), np.int64)
    rd = np.zeros((P, P), np.int64)
    for s in range(P):
        at = 0
        for d in range(P):
            sd[s, d] = at
            at += counts[s, d] + gap
    for d in range(P):
        at = gap
        for s in range(P):
            rd[d, s] = at
            at += counts[s, d] + gap
    with H.Comm(P, device=H.NO_DEVICE, chunk_bytes=chunk, validate=1) as c:
        H.hccl_alltoallv(c.handle, fake_bufs(P, 1 << 40), counts, sd, fake_bufs(P, 1 << 44), counts.T, rd, dt)
        info = c.last_program()
    assert info["bytes_written"] == int(counts.sum()) * ES[dt]


@SETTINGS
@given(st.integers(1, 64), st.integers(1, 300), st.integers(0, 5000), st.integers(0, 5000),
       st.sampled_from(["bf16", "fp16", "fp32", "int32"]), st.booleans(), st.booleans(), st.booleans())
def test_every_dynamic_exchange_validates(P, R, send_cap, recv_cap, dt, sd, rd, rc):
    meta = 1 << 47
    with H.Comm(P, device=H.NO_DEVICE, validate=1) as c:
        H.hccl_alltoallv_dynamic(c.handle, fake_bufs(P, 1 << 40), meta, meta + (1 << 20) if sd else None,
                                 fake_bufs(P, 1 << 44), meta + (3 << 20) if rc else None,
                                 meta + (2 << 20) if rd else None, R, send_cap, recv_cap, dt)
        info = c.last_program()
    assert info["num_descs"] == 1 and info["num_deps"] == 0 and info["num_tiles"] >= 1


@SETTINGS
@given(st.lists(st.tuples(st.sampled_from(["allreduce", "allgather", "reduce_scatter", "dynamic"]),
                          st.integers(1, 8), st.integers(0, 20000)), min_size=1, max_size=4))
def test_every_group_validates(calls):
    P = 8
    with H.Comm(P, device=H.NO_DEVICE, validate=1, algo="ring", fuse=0) as c:
        H.hccl_group_start(c.handle)
        ndyn = 0
        for k, (coll, _, n) in enumerate(calls):
            s, r = fake_bufs(P, (1 << 40) + k * (1 << 33)), fake_bufs(P, (1 << 44) + k * (1 << 33))
            if coll == "allreduce":
                H.hccl_allreduce(c.handle, s, r, n, "bf16")
            elif coll == "allgather":
                H.hccl_allgather(c.handle, s, r, n // P, "fp32")
            elif coll == "reduce_scatter":
                H.hccl_reduce_scatter(c.handle, s, r, n // P, "fp32")
            else:
                ndyn += 1
                H.hccl_alltoallv_dynamic(c.handle, s, (1 << 47) + k * (1 << 20), None, r, None, None, 4, 64, 512,
                                         "int32")
        if ndyn > 2:
            with pytest.raises(H.HcclError) as e:
                H.hccl_group_end(c.handle)
            assert e.value.code == 2
        else:
            H.hccl_group_end(c.handle)
