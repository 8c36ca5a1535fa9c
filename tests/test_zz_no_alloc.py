"""The allocation-free all-reduce (hccl_allreduce_noalloc) against hccl_allreduce.

hccl_allreduce_noalloc keeps its program image, dependency counters and FP32 partials in the
library's static workspace instead of device memory it allocates. Through the C ABI, each case
makes two calls in a row on one communicator, the second with a smaller input (so the second
call finds the workspace as the first left it), and every output element must equal what
hccl_allreduce writes for the same inputs, and the oracle's result. Guard bands around every
output must survive.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import Guarded, first_mismatch, same_bits, to_device
from workloads import normal_bf16, uniform_f32

pytestmark = pytest.mark.gpu

# label, ranks, element type, configuration, first and second element count, oracle order
CASES = [
    ("ring unfused bf16", 4, "bf16", dict(algo="ring", fuse=0, chunk_bytes=8192, phases="one"), 300_001, 70_003, {}),
    ("ring unfused bf16, a launch per level", 4, "bf16", dict(algo="ring", fuse=0, chunk_bytes=8192), 300_001,
     70_003, {}),
    ("two-level unfused bf16", 16, "bf16", dict(algo="two_level", group_size=4, fuse=0, chunk_bytes=16384,
                                                phases="one"), 200_000, 33_333, {"group": 4}),
    ("two-level fused bf16, copies in a second launch", 16, "bf16", dict(algo="two_level", group_size=4,
                                                                        phases="levels"), 200_000, 33_333, {"group": 4}),
    ("recursive halving unfused bf16", 8, "bf16", dict(algo="rhd", order="halving", fuse=0, phases="one"), 100_000,
     4_097, {"order": "halving"}),
    ("ring fused fp32", 8, "fp32", dict(algo="ring", chunk_bytes=65536), 1 << 20, 12_345, {}),
    ("one-step direct fp32", 8, "fp32", dict(algo="direct"), 1 << 14, 1000, {}),
]


def _inputs(P, n, dt, seed):
    return normal_bf16(P, n, std=1.0, seed=seed) if dt == "bf16" else uniform_f32(P, n, seed=seed)


def _want(x, dt, order):
    if order.get("order") == "halving":
        return oracle.allreduce_ordered(x, dt, order="halving")
    return oracle.allreduce(x, dt, group=order.get("group", 0))


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_allreduce_on_two_calls_second_smaller(case):
    label, P, dt, cfg, n1, n2, order = case
    with H.Comm(P, device=0, **cfg) as c:
        for k, n in enumerate((n1, n2)):
            print(f"noalloc: {label}, call {k + 1}, P={P} n={n}", flush=True)
            x = _inputs(P, n, dt, seed=700 + 10 * k + P)
            send = [to_device(x[r], dt) for r in range(P)]
            got = [Guarded(n, dt) for _ in range(P)]
            ref = [Guarded(n, dt) for _ in range(P)]
            H.hccl_allreduce_noalloc(c.handle, send, [g.view for g in got], n, dt)
            info = c.last_program()
            torch.cuda.synchronize()
            assert c.async_error() == 0
            H.hccl_allreduce(c.handle, send, [g.view for g in ref], n, dt)
            torch.cuda.synchronize()
            assert c.async_error() == 0
            if cfg.get("fuse") == 0 and P > 2:
                assert info["scratch_bytes"] > 0, info                            # partials used
                assert (info["num_deps"] > 0) == (cfg.get("phases") == "one"), info  # counters used
            if cfg.get("phases") == "levels" or (cfg.get("fuse") == 0 and "phases" not in cfg):
                assert info["num_phases"] > 1, info
            want = _want(x, dt, order)
            for r in range(P):
                a, b = got[r].result(), ref[r].result()
                assert same_bits(a, b, dt, nan_equal=False), f"rank {r} vs hccl_allreduce: {first_mismatch(a, b)}"
                assert same_bits(a, want[r], dt, nan_equal=False), f"rank {r} vs oracle: {first_mismatch(a, want[r])}"
                assert got[r].guards_intact(), f"rank {r}: guard band overwritten"


def test_noalloc_rejects_a_call_beyond_the_workspace_and_enqueues_nothing():
    # two-level unfused, 2 groups x 2^24 elements of FP32 partials = 128 MiB > 64 MiB
    P, n = 4, 1 << 24
    print("noalloc: beyond the workspace", flush=True)
    with H.Comm(P, device=0, algo="two_level", group_size=2, fuse=0) as c:
        send = [torch.zeros(n, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
        recv = [torch.full((n,), 3.0, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
        with pytest.raises(H.HcclError) as e:
            H.hccl_allreduce_noalloc(c.handle, send, recv, n, "bf16")
        assert e.value.code == 1 and "workspace" in str(e.value)
        torch.cuda.synchronize()
        assert all(bool((t == 3.0).all()) for t in recv)     # nothing ran
        assert c.async_error() == 0


def test_noalloc_refuses_groups_and_host_only_communicators():
    print("noalloc: refusals", flush=True)
    P, n = 2, 1000
    with H.Comm(P, device=0) as c:
        send = [torch.ones(n, dtype=torch.float32, device="cuda:0") for _ in range(P)]
        recv = [torch.empty(n, dtype=torch.float32, device="cuda:0") for _ in range(P)]
        with pytest.raises(H.HcclError) as e:
            with c.group():
                H.hccl_allreduce_noalloc(c.handle, send, recv, n, "fp32")
        assert e.value.code == 2
    with H.Comm(P, device=H.NO_DEVICE) as c:
        with pytest.raises(H.HcclError) as e:
            H.hccl_allreduce_noalloc(c.handle, [1 << 40, 2 << 40], [3 << 40, 4 << 40], n, "fp32")
        assert e.value.code == 1
