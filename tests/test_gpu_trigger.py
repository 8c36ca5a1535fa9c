"""GPU parity for device-triggered collectives (paper Section IV-B-3).

A collective is enqueued first, on a CU-masked stream, with a trigger: it occupies its CUs but
starts no step until a device word satisfies a comparison. The "compute" side, on a
non-blocking stream (so that nothing it does waits behind the waiting collective), then writes
the collective's inputs and finally the word. The outputs must be the
oracle's result over the inputs written after the launch (so the collective did wait), and the
completion word must hold its value once the collective is done.
"""
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import Guarded, MaskedStream, SideStream, first_mismatch, same_bits, to_device, to_host
from test_gpu_parity import inputs

pytestmark = pytest.mark.gpu


def words():
    return (torch.zeros(1, dtype=torch.int64, device="cuda:0"), torch.zeros(1, dtype=torch.int64, device="cuda:0"))


@pytest.mark.parametrize("algo,fuse", [("ring", 1), ("ring", 0), ("direct", 1)])
def test_prelaunched_allreduce_waits_for_its_inputs(algo, fuse):
    P, N = 8, 30011
    x = inputs(P, N, "bf16", 31)
    src = [to_device(x[r], "bf16") for r in range(P)]
    send = [torch.zeros(N, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
    outs = [Guarded(N, "bf16") for _ in range(P)]
    flag, done = words()
    print(f"triggered allreduce algo={algo} fuse={fuse}", flush=True)
    torch.cuda.synchronize()
    with MaskedStream(2) as s, SideStream() as cs, H.Comm(P, device=0, algo=algo, fuse=fuse,
                                                          chunk_bytes=8192) as c:
        with c.triggered(wait=(flag, "ge", 1), done=(done, 41)):
            H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, "bf16", stream=s)
        time.sleep(0.02)                       # the collective is resident and waiting by now
        with torch.cuda.stream(cs):
            for r in range(P):
                send[r].copy_(src[r])          # the compute side produces the inputs ...
            flag.fill_(1)                      # ... and then releases the collective
        cs.synchronize()
        s.synchronize()
        assert c.async_error() == 0
    assert int(done.item()) == 41
    want = oracle.allreduce(x, "bf16")
    for r in range(P):
        got = outs[r].result()
        assert same_bits(got, want[r], "bf16"), f"rank {r}: {first_mismatch(got, want[r])}"
        assert outs[r].guards_intact()


@pytest.mark.parametrize("cmp,value,flag_value", [("eq", 5, 5), ("ne", 0, 3), ("ge", 4, 4), ("gt", 4, 5),
                                                  ("le", 2, 2), ("lt", 9, 8)])
def test_every_comparator(cmp, value, flag_value):
    P, N = 4, 4099
    x = inputs(P, N, "fp32", 32)
    send = [to_device(x[r], "fp32") for r in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    flag, done = words()
    # start from a value that does not satisfy the comparison: above the threshold for "le" and
    # "lt", equal to it for "ne", zero otherwise
    flag.fill_(1 << 40 if cmp in ("le", "lt") else (value if cmp == "ne" else 0))
    torch.cuda.synchronize()
    print(f"trigger comparator {cmp} {value} <- {flag_value}", flush=True)
    with MaskedStream(2) as s, SideStream() as cs, H.Comm(P, device=0) as c:
        with c.triggered(wait=(flag, cmp, value), done=(done, 1)):
            H.hccl_allreduce(c.handle, send, recv, N, "fp32", stream=s)
        time.sleep(0.01)
        with torch.cuda.stream(cs):
            flag.fill_(flag_value)
        cs.synchronize()
        s.synchronize()
        assert c.async_error() == 0
    assert int(done.item()) == 1
    want = oracle.allreduce(x, "fp32")
    for r in range(P):
        assert same_bits(to_host(recv[r], "fp32"), want[r], "fp32")


def test_prelaunched_dynamic_alltoallv_reads_counts_written_after_launch():
    """Section V-F-2's pairing: a device-resident AllToAllv that is also device-triggered. The
    routing (counts and the sorted send rows) is produced after the exchange was enqueued."""
    P, R, S = 8, 64, 128
    cap = P * S
    x = inputs(P, S * R, "bf16", 33)
    src = [to_device(x[s], "bf16") for s in range(P)]
    send = [torch.zeros(S * R, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
    recv = [torch.zeros(cap * R, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
    rng = np.random.default_rng(8)
    counts = np.stack([rng.multinomial(S - 5, np.full(P, 1.0 / P)) for _ in range(P)])
    d_counts = torch.zeros(P * P, dtype=torch.int64, device="cuda:0")
    d_rc = torch.zeros(P * P, dtype=torch.int64, device="cuda:0")
    flag, done = words()
    torch.cuda.synchronize()
    host_counts = torch.from_numpy(counts.reshape(-1)).to("cuda:0")
    torch.cuda.synchronize()
    with MaskedStream(2) as s, SideStream() as cs, H.Comm(P, device=0) as c:
        with c.triggered(wait=(flag, "eq", 1), done=(done, 2)):
            c.alltoallv_dynamic(send, d_counts, recv, R, recvcounts=d_rc, stream=s)
        time.sleep(0.02)
        with torch.cuda.stream(cs):
            d_counts.copy_(host_counts)
            for r in range(P):
                send[r].copy_(src[r])
            flag.fill_(1)
        cs.synchronize()
        s.synchronize()
        assert c.async_error() == 0
    assert int(done.item()) == 2
    want = [np.zeros(cap * R, np.uint16) for _ in range(P)]
    ok, rc = oracle.alltoallv_dynamic([x[s] for s in range(P)], counts, want, R, S, cap)
    assert ok
    for d in range(P):
        assert np.array_equal(to_host(recv[d], "bf16"), want[d]), f"destination {d}"
    assert np.array_equal(d_rc.cpu().numpy().reshape(P, P), rc)


def test_completion_word_without_a_wait_and_for_a_group():
    P, M = 4, 3000
    x = inputs(P, M, "int32", 34)
    send = [to_device(x[r], "int32") for r in range(P)]
    ag = [torch.empty(P * M, dtype=torch.int32, device="cuda:0") for _ in range(P)]
    x2 = inputs(P, P * 100, "fp32", 35)
    send2 = [to_device(x2[r], "fp32") for r in range(P)]
    rs = [torch.empty(100, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    _, done = words()
    with H.Comm(P, device=0) as c:
        with c.triggered(done=(done, 9)):
            with c.group():
                c.allgather(send, ag)
                c.reduce_scatter(send2, rs)
        torch.cuda.synchronize()
        assert c.async_error() == 0
        assert int(done.item()) == 9
        # the trigger was consumed: the next call runs untriggered and leaves the word alone
        done.fill_(0)
        c.allgather(send, ag)
        torch.cuda.synchronize()
        assert int(done.item()) == 0
    want = oracle.allgather(x)
    for r in range(P):
        assert np.array_equal(to_host(ag[r], "int32"), want[r])
    want2 = oracle.reduce_scatter(x2, "fp32")
    for r in range(P):
        assert same_bits(to_host(rs[r], "fp32"), want2[r], "fp32")


def test_trigger_never_satisfied_times_out_and_moves_nothing():
    """The word is never written: every workgroup gives up after the communicator's (short)
    watchdog, the launch ends, nothing is written and the completion word stays unset."""
    P, N = 4, 5000
    x = inputs(P, N, "fp32", 36)
    send = [to_device(x[r], "fp32") for r in range(P)]
    outs = [Guarded(N, "fp32") for _ in range(P)]
    flag, done = words()
    with MaskedStream(2) as s, H.Comm(P, device=0, timeout_ms=50) as c:
        with c.triggered(wait=(flag, "eq", 1), done=(done, 1)):
            H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, "fp32", stream=s)
        s.synchronize()
        assert c.async_error() == 5
        assert "trigger" in H.hccl_get_last_error()
        # the communicator works again once the error was read
        H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, "fp32", stream=s)
        s.synchronize()
        assert c.async_error() == 0
    assert int(done.item()) == 0
    want = oracle.allreduce(x, "fp32")
    for r in range(P):
        assert same_bits(outs[r].result(), want[r], "fp32")


def test_compile_and_scratch_growth_while_a_triggered_packet_waits():
    """While a triggered all-reduce waits on its masked stream (holding those CUs), the same
    communicator compiles a new program, grows its scratch and runs an unfused ring
    reduce-scatter on another stream. That must finish before the trigger is released: nothing
    the library does then waits for every stream of the device (the upload goes on a stream of
    its own, the old scratch is kept instead of freed), and the dependent program drains on the
    CUs left to it (its tiles go by ticket). Then the trigger is released."""
    P, N, M = 8, 30011, 4001
    x = inputs(P, N, "bf16", 33)
    y = inputs(P, P * M, "bf16", 34)
    send = [to_device(x[r], "bf16") for r in range(P)]
    outs = [Guarded(N, "bf16") for _ in range(P)]
    ysend = [to_device(y[r], "bf16") for r in range(P)]
    small = [torch.empty(100, dtype=torch.bfloat16, device="cuda:0") for _ in range(P * 2)]
    youts = [Guarded(M, "bf16") for _ in range(P)]
    flag, done = words()
    torch.cuda.synchronize()
    print("trigger pending: compile, scratch growth and a dependent program on another stream", flush=True)
    with MaskedStream(2) as s, SideStream() as cs, H.Comm(P, device=0, chunk_bytes=8192, timeout_ms=10000) as c:
        c.set_config(algo="ring", fuse=0, chunk_bytes=8192, timeout_ms=10000, phases="one")
        H.hccl_allreduce(c.handle, small[:P], small[P:], 100, "bf16", stream=cs)   # a first, small scratch
        cs.synchronize()
        c.set_config(algo="ring", chunk_bytes=8192, timeout_ms=10000)
        with c.triggered(wait=(flag, "ge", 1), done=(done, 7)):
            H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, "bf16", stream=s)
        time.sleep(0.02)
        c.set_config(algo="ring", fuse=0, chunk_bytes=8192, timeout_ms=10000, phases="one")
        t0 = time.perf_counter()
        H.hccl_reduce_scatter(c.handle, ysend, [o.view for o in youts], M, "bf16", stream=cs)
        tickets = c.last_program()["tickets"]
        cs.synchronize()
        elapsed = time.perf_counter() - t0
        with torch.cuda.stream(cs):
            before = int(done.cpu())          # the triggered packet has not run yet
            flag.fill_(1)
        cs.synchronize()
        s.synchronize()
        assert c.async_error() == 0
    assert before == 0 and int(done.item()) == 7
    assert tickets == 1    # a dependent program while a triggered packet waits takes tiles by ticket
    assert elapsed < 2.0, f"the reduce-scatter took {elapsed:.2f} s while the trigger waited"
    want = oracle.allreduce(x, "bf16")
    for r in range(P):
        assert same_bits(outs[r].result(), want[r], "bf16") and outs[r].guards_intact()
    wrs = oracle.reduce_scatter(y, "bf16")
    for r in range(P):
        assert same_bits(youts[r].result(), wrs[r], "bf16") and youts[r].guards_intact()
