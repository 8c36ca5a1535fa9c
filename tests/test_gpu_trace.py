"""Per-tile trace (hcclConfig_t.trace, hccl_comm_trace): every tile of a traced launch leaves one
record, written by the wavefront the static schedule gives it, with consistent times, while the
results stay bit-exact against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import Guarded, same_bits, to_device
from program_interpreter import Program
from workloads import alltoallv_layout, normal_bf16, zipf_counts

pytestmark = pytest.mark.gpu


def _check_records(rec, khz, info, phase_tile=None):
    n = info["num_tiles"]
    assert rec.shape == (n,)
    assert (rec["start"] > 0).all(), "a tile left no record"
    assert (rec["done"] >= rec["ready"]).all()
    if not info["tickets"] and info["num_phases"] > 1:
        # one launch per phase, each static: wavefront w runs tiles b + w, b + w + W, ... of its
        # phase, and a phase starts after the previous one has ended
        for q in range(info["num_phases"]):
            lo, hi = int(phase_tile[q]), int(phase_tile[q + 1])
            W = int(rec["wave"][lo:hi].max()) + 1
            assert W <= info["workers"]
            assert np.array_equal(rec["wave"][lo:hi], np.arange(hi - lo, dtype=np.uint32) % W)
            if q:
                prev_end = (rec["start"][:lo].astype(np.int64) + rec["done"][:lo]).max()
                assert int(rec["start"][lo:hi].min()) >= prev_end
    elif not info["tickets"]:
        # static dispatch: wavefront w runs tiles w, w + W, ...
        assert np.array_equal(rec["wave"], np.arange(n, dtype=np.uint32) % info["workers"])
    else:
        # tickets: every wavefront takes its tiles in increasing order, one after the other
        assert (rec["wave"] < info["workers"]).all()
        for w in np.unique(rec["wave"]):
            mine = np.nonzero(rec["wave"] == w)[0]
            assert (np.diff(rec["start"][mine].astype(np.int64)) >= 0).all()
    assert ((rec["where"] >> 24) < 8).all()                   # XCC ids of the device
    span_us = (int((rec["start"] + rec["done"]).max()) - int(rec["start"].min())) * 1e3 / khz
    assert 0 < span_us < 1e6
    return span_us


@pytest.mark.parametrize("fuse,phases", [(0, "one"), (0, "auto"), (1, "auto")])
def test_traced_ring_allreduce_records_every_tile(fuse, phases):
    P, N = 4, 300_001
    print(f"trace: ring allreduce P={P} N={N} fuse={fuse} phases={phases}", flush=True)
    x = normal_bf16(P, N, seed=900 + fuse)
    with H.Comm(P, device=0, algo="ring", fuse=fuse, chunk_bytes=16384, trace=1, phases=phases) as c:
        send = [to_device(x[r], "bf16") for r in range(P)]
        out = [Guarded(N, "bf16") for _ in range(P)]
        c.allreduce(send, [o.view for o in out])
        torch.cuda.synchronize()
        assert c.async_error() == 0
        info = c.last_program()
        rec, khz = c.trace()
        phase_tile = Program(c.program_image()).phase_tile
    assert info["inline_launch"] == 0
    span = _check_records(rec, khz, info, phase_tile)
    want = oracle.allreduce(x, "bf16")
    for r in range(P):
        assert same_bits(out[r].result(), want[r], "bf16") and out[r].guards_intact()
    assert info["tickets"] == 0     # nothing else holds CUs: static dispatch
    if not fuse and phases == "one":
        assert (rec["ready"] > 0).any()   # a dependent step waits
    if not fuse and phases == "auto":
        assert info["num_phases"] == 2 * (P - 1) and info["num_deps"] == 0
    print(f"trace: {info['num_tiles']} tiles over {span:.1f} us", flush=True)


def test_trace_follows_the_last_launch_and_groups():
    P = 8
    counts = zipf_counts(P, 3000, 1.1, seed=11)
    rows, ids = alltoallv_layout(counts, 128), alltoallv_layout(counts, 1)
    rng = np.random.default_rng(12)
    rh = [rng.integers(0, 2 ** 16, int(rows["send_len"][s]), dtype=np.int64).astype(np.uint16) for s in range(P)]
    ih = [rng.integers(-2 ** 31, 2 ** 31, int(ids["send_len"][s]), dtype=np.int64).astype(np.int32) for s in range(P)]
    print("trace: grouped alltoallv, then a one-step allreduce", flush=True)
    with H.Comm(P, device=0, trace=1) as c:
        sr = [to_device(rh[s], "bf16") for s in range(P)]
        si = [to_device(ih[s], "int32") for s in range(P)]
        rr = [torch.zeros(int(rows["recv_len"][d]), dtype=torch.bfloat16, device="cuda:0") for d in range(P)]
        ri = [torch.zeros(int(ids["recv_len"][d]), dtype=torch.int32, device="cuda:0") for d in range(P)]
        with c.group():
            c.alltoallv(sr, rows["sendcounts"], rows["sdispls"], rr, rows["recvcounts"], rows["rdispls"])
            c.alltoallv(si, ids["sendcounts"], ids["sdispls"], ri, ids["recvcounts"], ids["rdispls"])
        torch.cuda.synchronize()
        g_info = c.last_program()
        g_rec, khz = c.trace()
        _check_records(g_rec, khz, g_info)
        x = np.random.default_rng(13).standard_normal((P, 5000)).astype(np.float32)
        send = [to_device(x[r], "fp32") for r in range(P)]
        recv = [torch.empty(5000, dtype=torch.float32, device="cuda:0") for _ in range(P)]
        c.allreduce(send, recv)       # one step: traced launches take the image path
        torch.cuda.synchronize()
        a_info = c.last_program()
        a_rec, khz = c.trace()
        assert a_info["inline_launch"] == 0 and a_rec.shape[0] == a_info["num_tiles"] != g_info["num_tiles"]
        _check_records(a_rec, khz, a_info)
        assert c.async_error() == 0
    want = oracle.allreduce(x, "fp32")
    assert same_bits(recv[3].cpu().numpy(), want[3], "fp32")
