"""GPU parity of the resident executor: work packets handed over through the host doorbell.

Every packet's outputs are compared bit for bit with the oracle after hccl_resident_wait. While
the executor runs nothing here waits for the whole device (it would wait for the executor
itself): inputs are written and read with stream-level synchronisation only.
"""
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import first_mismatch, same_bits, to_device, to_host
from test_gpu_parity import inputs

pytestmark = pytest.mark.gpu

IDLE_MS = 5000


def put(dst, bits, dt):
    dst.copy_(to_device(bits, dt))
    torch.cuda.current_stream().synchronize()


@pytest.mark.parametrize("algo,cfg,N", [("direct", {}, 16384), ("ring", dict(fuse=1), 100003),
                                        ("ring", dict(fuse=0), 50000), ("ring", dict(fuse=0, phases="one"), 50000),
                                        ("two_level", dict(group_size=4, fuse=0), 40000),
                                        ("two_level", dict(group_size=4, fuse=0, phases="one"), 40000)])
def test_resident_allreduce_packets_match_the_oracle(algo, cfg, N):
    P = 8
    print(f"resident allreduce algo={algo} cfg={cfg} N={N}", flush=True)
    xs = [inputs(P, N, "fp32", 100 + k) for k in range(3)]
    send = [torch.empty(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    order = "two_level" if algo == "two_level" else "ascending"
    with H.Comm(P, device=0, algo=algo, chunk_bytes=16384, **cfg) as c:
        for r in range(P):
            put(send[r], xs[0][r], "fp32")
        c.allreduce(send, recv)                  # compiles the program and sizes the scratch
        torch.cuda.synchronize()
        assert c.async_error() == 0
        phases = c.last_program()["num_phases"]
        with c.resident(idle_ms=IDLE_MS):
            for k in range(3):
                for r in range(P):
                    put(send[r], xs[k][r], "fp32")
                    recv[r].fill_(-1.0)
                torch.cuda.current_stream().synchronize()
                c.allreduce(send, recv)
                assert c.resident_seq() == (k + 1) * phases     # one packet per phase
                c.resident_wait()
                want = oracle.allreduce_ordered(xs[k], "fp32", order=order, group=cfg.get("group_size", 0))
                for r in range(P):
                    got = to_host(recv[r], "fp32")
                    assert same_bits(got, want[r], "fp32"), f"packet {k} rank {r}: {first_mismatch(got, want[r])}"


@pytest.mark.parametrize("phases", ["one", "auto"])
def test_resident_burst_wraps_the_doorbell_ring(phases):
    """150 calls submitted without waiting (more than the 64 slots: the call waits for a free
    slot), alternating two programs; a dependent program's counters must be clear for the next
    (in one launch), or every phase is a packet of its own."""
    P, N = 4, 30000
    x = inputs(P, N, "fp32", 110)
    send = [to_device(x[r], "fp32") for r in range(P)]
    out_a = [torch.zeros(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    out_b = [torch.zeros(N // P, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    print(f"resident burst of 150 calls, phases={phases}", flush=True)
    with H.Comm(P, device=0, algo="ring", fuse=0, chunk_bytes=8192, phases=phases) as c:
        c.allreduce(send, out_a)
        n_a = c.last_program()["num_phases"]
        c.reduce_scatter(send, out_b)
        n_b = c.last_program()["num_phases"]
        torch.cuda.synchronize()
        assert (n_a, n_b) == ((1, 1) if phases == "one" else (2 * (P - 1), P - 1))
        with c.resident(idle_ms=IDLE_MS):
            for k in range(150):
                if k % 2 == 0:
                    c.allreduce(send, out_a)
                else:
                    c.reduce_scatter(send, out_b)
            assert c.resident_seq() == 75 * (n_a + n_b)
            c.resident_wait(timeout_ms=10000)
        want = oracle.allreduce(x, "fp32")
        want_rs = oracle.reduce_scatter(x, "fp32")
        for r in range(P):
            assert same_bits(to_host(out_a[r], "fp32"), want[r], "fp32")
            assert same_bits(to_host(out_b[r], "fp32"), want_rs[r], "fp32")


def test_resident_group_of_alltoallv_and_allgather():
    P, R, D = 4, 200, 8
    rng = np.random.default_rng(12)
    counts = rng.multinomial(R, np.full(P, 1.0 / P), size=P) * D
    sd = np.concatenate([np.zeros((P, 1), np.int64), np.cumsum(counts, axis=1)[:, :-1]], axis=1)
    rd = np.concatenate([np.zeros((P, 1), np.int64), np.cumsum(counts.T, axis=1)[:, :-1]], axis=1)
    recv_len = counts.sum(axis=0)
    x = inputs(P, R * D, "bf16", 120)
    send = [to_device(x[r], "bf16") for r in range(P)]
    recv = [torch.zeros(int(recv_len[d]), dtype=torch.bfloat16, device="cuda:0") for d in range(P)]
    g_in = [to_device(x[r][:1000], "bf16") for r in range(P)]
    g_out = [torch.zeros(P * 1000, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
    print("resident group alltoallv + allgather", flush=True)

    def packet():
        with c.group():
            c.alltoallv(send, counts, sd, recv, counts.T, rd)
            c.allgather(g_in, g_out)

    with H.Comm(P, device=0) as c:
        packet()
        torch.cuda.synchronize()
        for t in recv + g_out:
            t.zero_()
        torch.cuda.synchronize()
        with c.resident(blocks=8, idle_ms=IDLE_MS):
            packet()
            c.resident_wait()
    want = [np.zeros(int(recv_len[d]), np.uint16) for d in range(P)]
    oracle.alltoallv([x[s] for s in range(P)], counts, sd, want, counts.T, rd)
    want_g = oracle.allgather(np.stack([x[r][:1000] for r in range(P)]))
    for d in range(P):
        assert np.array_equal(to_host(recv[d], "bf16"), want[d]), f"destination {d}"
        assert np.array_equal(to_host(g_out[d], "bf16"), want_g[d]), f"allgather rank {d}"


def test_resident_dynamic_exchange_reads_device_counts_per_packet():
    P, R, S = 8, 32, 80
    cap = P * S
    rng = np.random.default_rng(13)
    x = inputs(P, S * R, "int32", 130)
    send = [to_device(x[s], "int32") for s in range(P)]
    recv = [torch.empty(cap * R, dtype=torch.int32, device="cuda:0") for _ in range(P)]
    d_counts = torch.zeros(P * P, dtype=torch.int64, device="cuda:0")
    d_rc = torch.full((P * P,), -7, dtype=torch.int64, device="cuda:0")
    plans = [rng.multinomial(S, rng.dirichlet(np.full(P, 0.5)), size=P), np.zeros((P, P), np.int64)]
    bad = rng.multinomial(S, np.full(P, 1.0 / P), size=P)
    bad[3, 5] = -1                                        # a negative count: rejected, nothing moves
    plans += [bad, rng.multinomial(S // 3, np.full(P, 1.0 / P), size=P)]
    print("resident alltoallv_dynamic", flush=True)
    with H.Comm(P, device=0) as c:
        c.alltoallv_dynamic(send, d_counts, recv, R, recvcounts=d_rc)
        torch.cuda.synchronize()
        with c.resident(idle_ms=IDLE_MS):
            for k, counts in enumerate(plans):
                put(d_counts, counts.reshape(-1).astype(np.int64), "int64")
                for t in recv:
                    t.fill_(-1)
                torch.cuda.current_stream().synchronize()
                c.alltoallv_dynamic(send, d_counts, recv, R, recvcounts=d_rc)
                want = [np.full(cap * R, -1, np.int32) for _ in range(P)]
                accepted, want_rc = oracle.alltoallv_dynamic([x[s] for s in range(P)], counts, want, R, S, cap)
                if accepted:
                    c.resident_wait()
                else:
                    with pytest.raises(H.HcclError) as e:
                        c.resident_wait()
                    assert e.value.code == 1, str(e.value)
                assert np.array_equal(d_rc.cpu().numpy().reshape(P, P), want_rc), f"packet {k} recvcounts"
                for d in range(P):
                    assert np.array_equal(to_host(recv[d], "int32"), want[d]), f"packet {k} destination {d}"


def test_resident_compiles_new_shapes_and_refuses_what_it_cannot_run():
    P, N = 4, 8192
    x = inputs(P, N, "fp32", 140)
    send = [to_device(x[r], "fp32") for r in range(P)]
    recv = [torch.zeros(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    flag = torch.zeros(1, dtype=torch.int64, device="cuda:0")
    print("resident new shapes and refusals", flush=True)
    with H.Comm(P, device=0, algo="ring", fuse=0, chunk_bytes=4096) as c:
        with c.resident(idle_ms=IDLE_MS):
            # a new program without scratch is compiled on the host while the executor runs
            c.set_config(algo="direct", chunk_bytes=4096)
            c.allreduce(send, recv)
            assert c.last_program()["cache_hit"] == 0
            c.resident_wait()
            want = oracle.allreduce(x, "fp32")
            for r in range(P):
                assert same_bits(to_host(recv[r], "fp32"), want[r], "fp32")
            # one that needs scratch cannot grow it now
            c.set_config(algo="ring", fuse=0, chunk_bytes=4096)
            with pytest.raises(H.HcclError) as e:
                c.allreduce(send, recv)
            assert e.value.code == 2 and "scratch" in str(e.value)
            with pytest.raises(H.HcclError) as e:
                with c.triggered(wait=(flag, "ge", 1)):
                    c.set_config(algo="direct", chunk_bytes=4096)
                    c.allreduce(send, recv)
            assert e.value.code == 2
            assert c.async_error() == 1        # not available while the executor runs
        # stopped: calls launch on streams again
        c.set_config(algo="direct", chunk_bytes=4096)
        for t in recv:
            t.zero_()
        c.allreduce(send, recv)
        torch.cuda.synchronize()
        assert c.async_error() == 0
        for r in range(P):
            assert same_bits(to_host(recv[r], "fp32"), want[r], "fp32")


def test_resident_executor_ends_when_idle_and_restarts():
    P, N = 4, 4096
    send = [torch.ones(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    recv = [torch.zeros(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    print("resident idle end and restart", flush=True)
    with H.Comm(P, device=0) as c:
        H.hccl_resident_start(c.handle, 4, 100)
        time.sleep(0.5)                          # past the idle limit: the executor has ended
        with pytest.raises(H.HcclError) as e:
            c.allreduce(send, recv)
        assert e.value.code == 5 and "stopped" in str(e.value)
        H.hccl_resident_stop(c.handle)
        with c.resident(idle_ms=IDLE_MS):
            c.allreduce(send, recv)
            c.resident_wait()
        for r in range(P):
            assert bool(torch.all(recv[r] == P))
        with pytest.raises(H.HcclError) as e:
            H.hccl_resident_start(c.handle, 100000, 0)   # cannot all be resident at once
        assert e.value.code == 1


@pytest.mark.parametrize("blocks", [3, 32])
def test_resident_large_packets_where_the_relay_runs_tiles(blocks):
    """Packets with far more tiles than wavefronts, so the relay workgroup runs tiles of its own
    before it fetches the next packet; a direct and a dependent (unfused ring) program alternate,
    queued without waiting, and the last of each is checked. Two communicators run an executor
    each at the same time."""
    P, N = 8, 1 << 20
    x = inputs(P, N, "bf16", 150)
    send = [to_device(x[r], "bf16") for r in range(P)]
    out_a = [torch.zeros(N, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
    out_b = [torch.zeros(N, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
    print(f"resident large packets blocks={blocks}", flush=True)
    with H.Comm(P, device=0, algo="direct") as ca, H.Comm(P, device=0, algo="ring", fuse=0,
                                                          chunk_bytes=65536, phases="one") as cb:
        ca.allreduce(send, out_a)
        cb.allreduce(send, out_b)
        torch.cuda.synchronize()
        assert ca.last_program()["num_tiles"] > 32 * 4 and cb.last_program()["num_deps"] > 0
        for t in out_a + out_b:
            t.zero_()
        torch.cuda.synchronize()
        with ca.resident(blocks=blocks, idle_ms=IDLE_MS), cb.resident(blocks=blocks, idle_ms=IDLE_MS):
            for _ in range(6):
                ca.allreduce(send, out_a)
                cb.allreduce(send, out_b)
            ca.resident_wait(timeout_ms=20000)
            cb.resident_wait(timeout_ms=20000)
    want = oracle.allreduce(x, "bf16")
    for r in range(P):
        assert same_bits(to_host(out_a[r], "bf16"), want[r], "bf16"), f"direct rank {r}"
        assert same_bits(to_host(out_b[r], "bf16"), want[r], "bf16"), f"ring rank {r}"


def test_resident_wait_by_sequence_number():
    P, N = 4, 4096
    x = inputs(P, N, "fp32", 160)
    send = [to_device(x[r], "fp32") for r in range(P)]
    outs = [[torch.zeros(N, dtype=torch.float32, device="cuda:0") for _ in range(P)] for _ in range(5)]
    print("resident wait by sequence number", flush=True)
    with H.Comm(P, device=0) as c:
        for o in outs:
            c.allreduce(send, o)
        torch.cuda.synchronize()
        for o in outs:
            for t in o:
                t.zero_()
        torch.cuda.synchronize()
        with c.resident(blocks=4, idle_ms=IDLE_MS):
            for o in outs:
                c.allreduce(send, o)
            assert c.resident_seq() == 5
            c.resident_wait(seq=2)                   # the first two have completed, in order
            want = oracle.allreduce(x, "fp32")
            for o in outs[:2]:
                for r in range(P):
                    assert same_bits(to_host(o[r], "fp32"), want[r], "fp32")
            with pytest.raises(H.HcclError) as e:
                c.resident_wait(seq=6)               # never submitted
            assert e.value.code == 1
            c.resident_wait()
            for o in outs[2:]:
                for r in range(P):
                    assert same_bits(to_host(o[r], "fp32"), want[r], "fp32")
