"""Collectives captured into a HIP graph and replayed.

Once a program is compiled and uploaded, enqueueing it again on a capturing stream makes only
kernel launches: no allocation, no memset, no host synchronisation, no event. So after one
eager call a collective can be captured into a graph and replayed. Every replay is
checked against the oracle, with eager work between replays (new inputs written by torch,
host synchronisations); the cases cover an inline one-step launch, a fused program, a dependent
program whose counters are cleared in-kernel, a group of two calls, and a device-resident
exchange whose counts change between replays without the graph being captured again.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import first_mismatch, same_bits, to_device, to_host
from test_gpu_parity import inputs

pytestmark = pytest.mark.gpu

REPLAYS = 4


def capture(fn, stream):
    """One eager call (compiles and uploads the program), then a graph of the same call."""
    with torch.cuda.stream(stream):
        fn()
    stream.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        fn()
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("algo,fuse,N", [("direct", 1, 16384), ("ring", 1, 100003), ("ring", 0, 50000)])
def test_captured_allreduce_replays_match_the_oracle(algo, fuse, N):
    P = 8
    print(f"graph allreduce algo={algo} fuse={fuse} N={N}", flush=True)
    xs = [inputs(P, N, "fp32", 60 + k) for k in range(REPLAYS)]
    send = [to_device(xs[0][r], "fp32") for r in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    side = torch.cuda.Stream()
    with H.Comm(P, device=0, algo=algo, fuse=fuse, chunk_bytes=16384) as c:
        g = capture(lambda: c.allreduce(send, recv, stream=side), side)
        for k in range(REPLAYS):
            for r in range(P):
                send[r].copy_(to_device(xs[k][r], "fp32"))
                recv[r].fill_(-1.0)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert c.async_error() == 0
            want = oracle.allreduce(xs[k], "fp32")
            for r in range(P):
                got = to_host(recv[r], "fp32")
                assert same_bits(got, want[r], "fp32"), f"replay {k} rank {r}: {first_mismatch(got, want[r])}"


def test_captured_group_of_two_alltoallv_calls():
    P, R, D = 4, 300, 16
    rng = np.random.default_rng(5)
    counts = rng.multinomial(R, np.full(P, 1.0 / P), size=P) * D          # [src, dst] elements
    sd = np.concatenate([np.zeros((P, 1), np.int64), np.cumsum(counts, axis=1)[:, :-1]], axis=1)
    rd = np.concatenate([np.zeros((P, 1), np.int64), np.cumsum(counts.T, axis=1)[:, :-1]], axis=1)
    recv_len = counts.sum(axis=0)
    print(f"graph group of two alltoallv P={P} rows={R}", flush=True)
    xs = [inputs(P, R * D, "bf16", 70 + k) for k in range(REPLAYS)]
    send = [to_device(xs[0][r], "bf16") for r in range(P)]
    recv_a = [torch.empty(int(recv_len[d]), dtype=torch.bfloat16, device="cuda:0") for d in range(P)]
    recv_b = [torch.empty(int(recv_len[d]), dtype=torch.bfloat16, device="cuda:0") for d in range(P)]
    side = torch.cuda.Stream()
    with H.Comm(P, device=0) as c:
        def step():
            with c.group():
                c.alltoallv(send, counts, sd, recv_a, counts.T, rd, stream=side)
                c.alltoallv(send, counts, sd, recv_b, counts.T, rd, stream=side)

        g = capture(step, side)
        for k in range(REPLAYS):
            for r in range(P):
                send[r].copy_(to_device(xs[k][r], "bf16"))
                recv_a[r].fill_(0)
                recv_b[r].fill_(0)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert c.async_error() == 0
            want = [np.zeros(int(recv_len[d]), np.uint16) for d in range(P)]
            oracle.alltoallv([xs[k][s] for s in range(P)], counts, sd, want, counts.T, rd)
            for d in range(P):
                assert np.array_equal(to_host(recv_a[d], "bf16"), want[d]), f"replay {k} destination {d}"
                assert np.array_equal(to_host(recv_b[d], "bf16"), want[d]), f"replay {k} destination {d}"


def test_captured_dynamic_exchange_follows_device_counts():
    """The graph is captured once; each replay reads the count matrix that device memory holds
    at that moment, including an all-zero one and one the exchange must reject."""
    P, R, S = 8, 64, 96
    cap = P * S
    rng = np.random.default_rng(11)
    x = inputs(P, S * R, "int32", 80)
    send = [to_device(x[s], "int32") for s in range(P)]
    recv = [torch.empty(cap * R, dtype=torch.int32, device="cuda:0") for _ in range(P)]
    d_counts = torch.zeros(P * P, dtype=torch.int64, device="cuda:0")
    d_rc = torch.full((P * P,), -7, dtype=torch.int64, device="cuda:0")
    side = torch.cuda.Stream()
    print(f"graph alltoallv_dynamic P={P} rows={R}", flush=True)
    plans = [rng.multinomial(S, rng.dirichlet(np.full(P, 0.5)), size=P),
             np.zeros((P, P), np.int64),
             rng.multinomial(S // 2, np.full(P, 1.0 / P), size=P)]
    over = rng.multinomial(S, np.full(P, 1.0 / P), size=P)
    over[0, 0] = S + 1                                     # row 0 exceeds the send capacity
    plans.append(over)
    with H.Comm(P, device=0) as c:
        g = capture(lambda: c.alltoallv_dynamic(send, d_counts, recv, R, recvcounts=d_rc, stream=side), side)
        for k, counts in enumerate(plans):
            d_counts.copy_(torch.from_numpy(counts.reshape(-1).astype(np.int64)).to("cuda:0"))
            for t in recv:
                t.fill_(-1)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            want = [np.full(cap * R, -1, np.int32) for _ in range(P)]
            accepted, want_rc = oracle.alltoallv_dynamic([x[s] for s in range(P)], counts, want, R, S, cap)
            err = c.async_error()
            assert (err == 0) == accepted, f"replay {k}: error {err}, oracle accepted={accepted}"
            assert np.array_equal(d_rc.cpu().numpy().reshape(P, P), want_rc), f"replay {k} recvcounts"
            for d in range(P):
                assert np.array_equal(to_host(recv[d], "int32"), want[d]), f"replay {k} destination {d}"


def test_first_call_under_capture_is_refused_and_enqueues_nothing():
    P, N = 4, 4096
    send = [torch.ones(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    recv = [torch.zeros(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    side = torch.cuda.Stream()
    print("graph first call under capture", flush=True)
    with H.Comm(P, device=0) as c:
        g = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            with pytest.raises(H.HcclError) as e:
                c.allreduce(send, recv, stream=side)
        assert e.value.code == 2 and "outside the capture" in str(e.value)
        torch.cuda.synchronize()
        assert all(int(torch.count_nonzero(r)) == 0 for r in recv)
        c.allreduce(send, recv, stream=side)          # the same call outside a capture compiles and runs
        side.synchronize()
        assert all(bool(torch.all(r == P)) for r in recv)


def test_graph_outlives_eviction_of_its_program_and_scratch_growth():
    """A graph keeps the image, counters and scratch it captured: evicting its program from the
    cache (64 programs) and growing the scratch afterwards must not free them."""
    P, N = 8, 20000
    x = inputs(P, N, "fp32", 90)
    send = [to_device(x[r], "fp32") for r in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    side = torch.cuda.Stream()
    print("graph after eviction and scratch growth", flush=True)
    with H.Comm(P, device=0, algo="ring", fuse=0, chunk_bytes=16384) as c:
        g = capture(lambda: c.allreduce(send, recv, stream=side), side)
        assert c.last_program()["scratch_bytes"] > 0
        big = [torch.zeros(N + 80, dtype=torch.float32, device="cuda:0") for _ in range(P)]
        big_out = [torch.empty_like(b) for b in big]
        for extra in range(1, 80):            # 79 new programs, each with a larger scratch
            c.allreduce([b[:N + extra] for b in big], [o[:N + extra] for o in big_out], stream=side)
        side.synchronize()
        want = oracle.allreduce(x, "fp32")
        for k in range(2):
            for r in range(P):
                recv[r].fill_(-1.0)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert c.async_error() == 0
            for r in range(P):
                got = to_host(recv[r], "fp32")
                assert same_bits(got, want[r], "fp32"), f"replay {k} rank {r}: {first_mismatch(got, want[r])}"
