"""GPU parity of dependent programs under both ways of handing tiles to wavefronts.

By default programs take tiles statically (wavefront w runs tiles w, w + W, ...) and dependent
ones by atomic ticket while a waiting executor holds CUs; HCCL_DISPATCH=static makes every
program static, HCCL_DISPATCH=dynamic every program ticketed, and HCCL_INLINE=0 sends one-step
programs through the device image too.
Each mode must give the oracle's bits, launch after launch (the counters are cleared at the end
of every launch).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import Guarded, first_mismatch, same_bits, to_device, to_host
from test_gpu_parity import inputs

pytestmark = pytest.mark.gpu

SMALL = dict(chunk_bytes=4096, tile_bytes=4096)


@pytest.fixture(params=["auto", "static", "tickets", "no_inline"])
def mode(request, monkeypatch):
    if request.param == "static":
        monkeypatch.setenv("HCCL_DISPATCH", "static")
    if request.param == "tickets":
        monkeypatch.setenv("HCCL_DISPATCH", "dynamic")
    if request.param == "no_inline":
        monkeypatch.setenv("HCCL_INLINE", "0")
    return request.param


@pytest.mark.parametrize("phases", ["one", "auto"])
@pytest.mark.parametrize("algo,cfg", [("ring", dict(fuse=0)), ("two_level", dict(group_size=4, fuse=0)),
                                      ("rhd", dict(order="halving", fuse=0)), ("direct", {})])
def test_allreduce_repeated_launches(mode, algo, cfg, phases):
    P, N = 8, 12345
    x = inputs(P, N, "bf16", 21)
    cfg = dict(cfg, phases=phases)
    print(f"dispatch={mode} allreduce algo={algo} cfg={cfg}", flush=True)
    want = oracle.allreduce_ordered(x, "bf16", order=cfg.get("order", "two_level" if algo == "two_level" else
                                                           "ascending"), group=cfg.get("group_size", 0))
    with H.Comm(P, device=0, algo=algo, **cfg, **SMALL) as c:
        send = [to_device(x[r], "bf16") for r in range(P)]
        outs = [Guarded(N, "bf16") for _ in range(P)]
        for it in range(4):
            for o in outs:
                o.view.fill_(0)
            H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, "bf16")
            torch.cuda.synchronize()
            assert c.async_error() == 0
            for r in range(P):
                got = outs[r].result()
                assert same_bits(got, want[r], "bf16"), f"launch {it} rank {r}: {first_mismatch(got, want[r])}"
                assert outs[r].guards_intact()


def test_dynamic_alltoallv_repeated_launches(mode):
    P, R, S = 8, 16, 64
    cap = P * S
    x = inputs(P, S * R, "int32", 22)
    send = [to_device(x[s], "int32") for s in range(P)]
    recv = [torch.empty(cap * R, dtype=torch.int32, device="cuda:0") for _ in range(P)]
    d_counts = torch.zeros(P * P, dtype=torch.int64, device="cuda:0")
    rng = np.random.default_rng(3)
    print(f"dispatch={mode} alltoallv_dynamic", flush=True)
    with H.Comm(P, device=0) as c:
        run = c.bind_alltoallv_dynamic(send, d_counts, recv, R)
        for it in range(4):
            counts = np.stack([rng.multinomial(S - it, np.full(P, 1.0 / P)) for _ in range(P)])
            d_counts.copy_(torch.from_numpy(counts.reshape(-1)).to("cuda:0"))
            for t in recv:
                t.fill_(-1)
            run()
            torch.cuda.synchronize()
            assert c.async_error() == 0
            want = [np.full(cap * R, -1, np.int32) for _ in range(P)]
            assert oracle.alltoallv_dynamic([x[s] for s in range(P)], counts, want, R, S, cap)[0]
            for d in range(P):
                assert np.array_equal(to_host(recv[d], "int32"), want[d]), f"launch {it} destination {d}"


@pytest.mark.parametrize("phases", ["one", "auto"])
def test_triggered_dependent_program(mode, phases):
    """A pre-launched unfused ring all-reduce (dependent steps, waited for on the device or run
    as one launch per level behind the first) released by a device word, in every dispatch mode."""
    import time

    from gpu_helpers import MaskedStream, SideStream

    P, N = 4, 20000
    x = inputs(P, N, "fp32", 23)
    src = [to_device(x[r], "fp32") for r in range(P)]
    send = [torch.zeros(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    recv = [torch.empty(N, dtype=torch.float32, device="cuda:0") for _ in range(P)]
    flag = torch.zeros(1, dtype=torch.int64, device="cuda:0")
    done = torch.zeros(1, dtype=torch.int64, device="cuda:0")
    torch.cuda.synchronize()
    print(f"dispatch={mode} triggered unfused ring phases={phases}", flush=True)
    with MaskedStream(2) as s, SideStream() as cs, H.Comm(P, device=0, algo="ring", fuse=0, phases=phases,
                                                          **SMALL) as c:
        with c.triggered(wait=(flag, "eq", 3), done=(done, 4)):
            H.hccl_allreduce(c.handle, send, recv, N, "fp32", stream=s)
        time.sleep(0.01)
        with torch.cuda.stream(cs):
            for r in range(P):
                send[r].copy_(src[r])
            flag.fill_(3)
        cs.synchronize()
        s.synchronize()
        assert c.async_error() == 0
    assert int(done.item()) == 4
    want = oracle.allreduce(x, "fp32")
    for r in range(P):
        assert same_bits(to_host(recv[r], "fp32"), want[r], "fp32")


@pytest.mark.parametrize("max_workers", [0, 4, 100])
@pytest.mark.parametrize("algo", ["direct", "ring"])
def test_grid_of_programs_that_never_wait(algo, max_workers):
    """A launch with no dependency inside it gets one wavefront per tile (max_workers = 0);
    a capped grid makes every wavefront run many tiles in turn. Same bits either way."""
    from test_gpu_parity import run_allreduce, run_alltoallv, run_reduce_scatter
    from workloads import zipf_counts

    cfg = dict(algo=algo, fuse=1, chunk_bytes=65536, tile_bytes=4096, max_workers=max_workers)
    info = run_allreduce(8, 300001, "bf16", **cfg)
    assert info["num_phases"] == 1
    if max_workers == 0:
        assert info["num_tiles"] <= info["workers"] < info["num_tiles"] + 4
    else:
        assert info["workers"] == max_workers
    run_reduce_scatter(8, 70001, "fp32", **cfg)
    run_alltoallv(8, zipf_counts(8, 3000, 1.1, seed=5), 129, "bf16", max_workers=max_workers)


def test_triggered_launch_keeps_a_grid_the_cus_hold():
    """A triggered launch holds its workgroups at the trigger, so its grid stays within what the
    CUs hold at once; the same program launched untriggered gets one wavefront per tile. Both
    give the oracle's bits (the trigger word is already set: nothing waits)."""
    P, N = 8, 1 << 22  # 4 KiB tiles: 8 192 tiles, more than the chip holds at once
    x = inputs(P, N, "bf16", 24)
    want = oracle.allreduce(x, "bf16")
    flag = torch.ones(1, dtype=torch.int64, device="cuda:0")
    print("dispatch: triggered against untriggered grid", flush=True)
    with H.Comm(P, device=0, algo="direct", tile_bytes=4096) as c:
        send = [to_device(x[r], "bf16") for r in range(P)]
        for triggered in (False, True):
            recv = [torch.empty(N, dtype=torch.bfloat16, device="cuda:0") for _ in range(P)]
            if triggered:
                with c.triggered(wait=(flag, "eq", 1)):
                    c.allreduce(send, recv)
            else:
                c.allreduce(send, recv)
            torch.cuda.synchronize()
            assert c.async_error() == 0
            info = c.last_program()
            if triggered:
                assert 0 < info["workers"] < info["num_tiles"]
            else:
                assert info["workers"] >= info["num_tiles"]
            for r in range(P):
                got = to_host(recv[r], "bf16")
                assert same_bits(got, want[r], "bf16"), f"triggered={triggered} rank {r}: {first_mismatch(got, want[r])}"
