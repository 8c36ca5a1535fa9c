"""GPU parity: the HIP executor against the CPU oracle, bit for bit, through the C-ABI.

Inputs come from the seeded generators; expected values come from the oracle only. Sizes span
several tiles (small tiles are forced where needed) and ragged tails; every output buffer has
poison guard bands that must survive.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_00358_amd as H
from gpu_helpers import GUARD, Guarded, same_bits, first_mismatch, to_device, to_host
from workloads import alltoallv_layout, normal_bf16, normal_f32, row_ids_int32, uniform_f32, zipf_counts

pytestmark = pytest.mark.gpu

DT_ES = {"bf16": 2, "fp16": 2, "fp32": 4, "int32": 4}


def inputs(P, N, dt, seed):
    if dt == "fp32":
        return uniform_f32(P, N, seed=seed)
    if dt == "bf16":
        return normal_bf16(P, N, std=2.0, seed=seed)
    if dt == "fp16":
        return normal_f32(P, N, std=8.0, seed=seed).astype(np.float16).view(np.uint16)
    rng = np.random.default_rng(seed)
    return rng.integers(-2 ** 31, 2 ** 31, size=(P, N), dtype=np.int64).astype(np.int32)


def run_allreduce(P, N, dt, op="sum", in_place=False, seed=0, **cfg):
    x = inputs(P, N, dt, seed)
    print(f"allreduce P={P} N={N} dt={dt} op={op} in_place={in_place} cfg={cfg}", flush=True)
    with H.Comm(P, device=0, **cfg) as c:
        if in_place:
            bufs = [Guarded(N, dt, fill=x[r]) for r in range(P)]
            H.hccl_allreduce(c.handle, [b.view for b in bufs], [b.view for b in bufs], N, dt, op)
            outs = bufs
        else:
            send = [to_device(x[r], dt) for r in range(P)]
            outs = [Guarded(N, dt) for _ in range(P)]
            H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, dt, op)
        torch.cuda.synchronize()
        assert c.async_error() == 0
        info = c.last_program()
    want = oracle.allreduce(x, dt, op=op, group=cfg.get("group_size", 0) if cfg.get("algo") == "two_level" else 0)
    for r in range(P):
        got = outs[r].result()
        assert same_bits(got, want[r], dt), f"rank {r}: {first_mismatch(got, want[r])}"
        assert outs[r].guards_intact(), f"rank {r}: guard band overwritten"
    return info


@pytest.mark.parametrize("dt", ["fp32", "bf16", "fp16", "int32"])
@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("algo,fuse", [("direct", 1), ("ring", 1), ("ring", 0)])
def test_allreduce_matches_oracle(dt, P, algo, fuse):
    # 12345 elements with 4 KiB tiles: many tiles, a ragged vector tail and single elements
    run_allreduce(P, 12345, dt, algo=algo, fuse=fuse, chunk_bytes=8192, tile_bytes=4096)


@pytest.mark.parametrize("N", [1, 7, 8, 9, 511, 513, 4096])
def test_allreduce_small_and_ragged_sizes(N):
    run_allreduce(4, N, "bf16", algo="ring", fuse=1, tile_bytes=4096)
    run_allreduce(3, N, "fp32", algo="ring", fuse=0, chunk_bytes=256, tile_bytes=4096)


@pytest.mark.parametrize("fuse", [0, 1])
@pytest.mark.parametrize("dt", ["bf16", "fp32"])
def test_allreduce_in_place(fuse, dt):
    run_allreduce(5, 20011, dt, in_place=True, algo="ring", fuse=fuse, chunk_bytes=4096, tile_bytes=4096)


@pytest.mark.parametrize("op", ["max", "min"])
@pytest.mark.parametrize("dt", ["fp32", "bf16", "int32"])
@pytest.mark.parametrize("fuse", [0, 1])
def test_allreduce_max_min(op, dt, fuse):
    run_allreduce(6, 9999, dt, op=op, algo="ring", fuse=fuse, chunk_bytes=4096, tile_bytes=4096)


@pytest.mark.parametrize("L,G", [(4, 4), (8, 8), (2, 3), (1, 4), (4, 1)])
@pytest.mark.parametrize("fuse", [0, 1])
def test_two_level_allreduce_matches_tree_order_oracle(L, G, fuse):
    run_allreduce(L * G, 20000, "bf16", algo="two_level", group_size=L, fuse=fuse, chunk_bytes=8192,
                  tile_bytes=8192)


def run_reduce_scatter(P, M, dt, op="sum", seed=1, **cfg):
    x = inputs(P, P * M, dt, seed)
    print(f"reduce_scatter P={P} M={M} dt={dt} cfg={cfg}", flush=True)
    with H.Comm(P, device=0, **cfg) as c:
        send = [to_device(x[r], dt) for r in range(P)]
        outs = [Guarded(M, dt) for _ in range(P)]
        H.hccl_reduce_scatter(c.handle, send, [o.view for o in outs], M, dt, op)
        torch.cuda.synchronize()
        assert c.async_error() == 0
    want = oracle.reduce_scatter(x, dt, op=op)
    for r in range(P):
        got = outs[r].result()
        assert same_bits(got, want[r], dt), f"rank {r}: {first_mismatch(got, want[r])}"
        assert outs[r].guards_intact()


@pytest.mark.parametrize("dt", ["fp32", "bf16", "fp16", "int32"])
@pytest.mark.parametrize("P", [1, 2, 5, 8])
@pytest.mark.parametrize("algo,fuse", [("direct", 1), ("ring", 1), ("ring", 0)])
def test_reduce_scatter_matches_oracle(dt, P, algo, fuse):
    run_reduce_scatter(P, 3001, dt, algo=algo, fuse=fuse, chunk_bytes=2048, tile_bytes=4096)


def run_allgather(P, M, dt, seed=2, **cfg):
    x = inputs(P, M, dt, seed)
    print(f"allgather P={P} M={M} dt={dt} cfg={cfg}", flush=True)
    with H.Comm(P, device=0, **cfg) as c:
        send = [to_device(x[r], dt) for r in range(P)]
        outs = [Guarded(P * M, dt) for _ in range(P)]
        H.hccl_allgather(c.handle, send, [o.view for o in outs], M, dt)
        torch.cuda.synchronize()
        assert c.async_error() == 0
    want = oracle.allgather(x)
    for r in range(P):
        got = outs[r].result()
        assert np.array_equal(got.view(np.uint8), want[r].view(np.uint8)), f"rank {r}"
        assert outs[r].guards_intact()


@pytest.mark.parametrize("dt", ["bf16", "fp32"])
@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("M", [1, 5, 1000, 40001])
@pytest.mark.parametrize("algo,fuse", [("direct", 1), ("ring", 0)])
def test_allgather_matches_oracle(dt, P, M, algo, fuse):
    run_allgather(P, M, dt, algo=algo, fuse=fuse, chunk_bytes=8192, tile_bytes=4096)


def run_alltoallv(P, counts, elems_per_row, dt, seed=3, gap=0, **cfg):
    lay = alltoallv_layout(counts, elems_per_row)
    rdispls = lay["rdispls"].copy()
    recv_len = lay["recv_len"].copy()
    if gap:
        # receive blocks separated by `gap` untouched elements
        for d in range(P):
            off = gap
            for s in range(P):
                rdispls[d, s] = off
                off += lay["recvcounts"][d, s] + gap
            recv_len[d] = off
    rng = np.random.default_rng(seed)
    send_host = []
    for s in range(P):
        n = int(lay["send_len"][s])
        if dt == "int32":
            send_host.append(rng.integers(-2 ** 31, 2 ** 31, size=n, dtype=np.int64).astype(np.int32))
        else:
            send_host.append(rng.integers(0, 2 ** 16, size=n, dtype=np.int64).astype(np.uint16))
    print(f"alltoallv P={P} rows={counts.sum()} elems/row={elems_per_row} dt={dt} gap={gap} cfg={cfg}", flush=True)
    with H.Comm(P, device=0, **cfg) as c:
        send = [to_device(send_host[s], dt) for s in range(P)]
        outs = [Guarded(int(recv_len[d]), dt) for d in range(P)]
        H.hccl_alltoallv(c.handle, send, lay["sendcounts"], lay["sdispls"], [o.view for o in outs],
                         lay["recvcounts"], rdispls, dt)
        torch.cuda.synchronize()
        assert c.async_error() == 0
    expect = [o.host_init[64:64 + o.n].copy() for o in outs]
    oracle.alltoallv(send_host, lay["sendcounts"], lay["sdispls"], expect, lay["recvcounts"], rdispls)
    for d in range(P):
        got = outs[d].result()
        assert np.array_equal(got.view(np.uint8), expect[d].view(np.uint8)), f"dst {d}"
        assert outs[d].guards_intact()


@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("gap", [0, 3])
def test_alltoallv_embedding_rows_and_ids(P, gap):
    counts = zipf_counts(P, 3000, 1.1, seed=P)
    run_alltoallv(P, counts, 128, "bf16", gap=gap, chunk_bytes=65536, tile_bytes=16384)
    run_alltoallv(P, counts, 1, "int32", gap=gap, chunk_bytes=4096, tile_bytes=4096)


def test_alltoallv_zero_blocks_and_odd_row_widths():
    P = 5
    rng = np.random.default_rng(7)
    counts = rng.integers(0, 40, size=(P, P))
    counts[0, :] = 0
    counts[:, 3] = 0
    for elems in (1, 3, 7, 8, 9):
        run_alltoallv(P, counts, elems, "bf16", gap=1, chunk_bytes=512, tile_bytes=4096)
        run_alltoallv(P, counts, elems, "int32", gap=2, chunk_bytes=512, tile_bytes=4096)


def test_special_values_follow_the_oracle():
    P, N = 4, 4096
    rng = np.random.default_rng(11)
    specials = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, -1e-45, 1.17549435e-38,
                         3.4028235e38, -3.4028235e38, 65504.0, 65520.0, 6e-8, 1.0, -1.0], np.float32)
    x32 = specials[rng.integers(0, specials.size, size=(P, N))]
    print("special values fp32/bf16/fp16", flush=True)
    for dt, bits in (("fp32", x32), ("bf16", oracle.f32_to_bf16(x32)), ("fp16", oracle.f32_to_f16(x32))):
        with H.Comm(P, device=0, algo="direct", tile_bytes=4096) as c:
            send = [to_device(bits[r], dt) for r in range(P)]
            outs = [Guarded(N, dt) for _ in range(P)]
            H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, dt)
            torch.cuda.synchronize()
        want = oracle.allreduce(bits, dt)
        for r in range(P):
            got = outs[r].result()
            assert same_bits(got, want[r], dt), f"{dt} rank {r}: {first_mismatch(got, want[r])}"


def test_fp16_rounding_boundaries_of_the_hardware_conversion():
    # sums that land on fp16 ties, overflow thresholds and subnormals
    P = 2
    rng = np.random.default_rng(12)
    halves = rng.integers(0, 1 << 16, size=(P, 1 << 16)).astype(np.uint16)
    halves[0, :] = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    with H.Comm(P, device=0, algo="direct") as c:
        send = [to_device(halves[r], "fp16") for r in range(P)]
        outs = [Guarded(1 << 16, "fp16") for _ in range(P)]
        H.hccl_allreduce(c.handle, send, [o.view for o in outs], 1 << 16, "fp16")
        torch.cuda.synchronize()
    want = oracle.allreduce(halves, "fp16")
    got = outs[0].result()
    assert same_bits(got, want[0], "fp16"), first_mismatch(got, want[0])


def test_repeated_launches_of_a_dependent_program_reset_their_counters():
    # the unfused ring in one launch uses per-tile counters; ten launches in a row must all be right
    P, N = 8, 65536
    x = inputs(P, N, "bf16", 21)
    with H.Comm(P, device=0, algo="ring", fuse=0, chunk_bytes=16384, tile_bytes=8192, phases="one") as c:
        send = [to_device(x[r], "bf16") for r in range(P)]
        outs = [Guarded(N, "bf16") for _ in range(P)]
        want = oracle.allreduce(x, "bf16")
        for it in range(10):
            for o in outs:
                o.view.zero_()
            H.hccl_allreduce(c.handle, send, [o.view for o in outs], N, "bf16")
            torch.cuda.synchronize()
            assert c.async_error() == 0
            for r in range(P):
                assert same_bits(outs[r].result(), want[r], "bf16"), f"launch {it} rank {r}"


@pytest.mark.parametrize("phases", ["one", "auto"])
def test_launches_on_two_streams_are_ordered(phases):
    P, N = 4, 100000
    x = inputs(P, N, "fp32", 22)
    want = oracle.allreduce(x, "fp32")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    with H.Comm(P, device=0, algo="ring", fuse=0, chunk_bytes=16384, tile_bytes=8192, phases=phases) as c:
        send = [to_device(x[r], "fp32") for r in range(P)]
        o1 = [Guarded(N, "fp32") for _ in range(P)]
        o2 = [Guarded(N, "fp32") for _ in range(P)]
        torch.cuda.synchronize()
        H.hccl_allreduce(c.handle, send, [o.view for o in o1], N, "fp32", stream=s1)
        H.hccl_allreduce(c.handle, send, [o.view for o in o2], N, "fp32", stream=s2)
        torch.cuda.synchronize()
        assert c.async_error() == 0
    for r in range(P):
        assert same_bits(o1[r].result(), want[r], "fp32")
        assert same_bits(o2[r].result(), want[r], "fp32")


@pytest.mark.parametrize("dt", ["fp32", "bf16", "fp16", "int32"])
@pytest.mark.parametrize("P,N", [(8, 1 << 14), (3, 1000), (1, 77), (64, 4099)])
def test_single_step_programs_travel_inline(dt, P, N):
    info = run_allreduce(P, N, dt, algo="direct")
    assert info["inline_launch"] == 1 and info["num_descs"] == 1


@pytest.mark.parametrize("op", ["max", "min"])
def test_single_step_inline_max_min_and_misaligned_views(op):
    # a buffer view that is 4-byte but not 16-byte aligned takes the element path inline
    P, N = 4, 3001
    x = inputs(P, N + 1, "fp32", 30)
    with H.Comm(P, device=0, algo="direct") as c:
        send_full = [to_device(x[r], "fp32") for r in range(P)]
        send = [t[1:] for t in send_full]
        outs = [Guarded(N + 1, "fp32") for _ in range(P)]
        H.hccl_allreduce(c.handle, send, [o.view[1:] for o in outs], N, "fp32", op)
        torch.cuda.synchronize()
        assert c.last_program()["inline_launch"] == 1
    want = oracle.allreduce(np.ascontiguousarray(x[:, 1:]), "fp32", op=op)
    for r in range(P):
        got = outs[r].result()[1:]
        assert same_bits(got, want[r], "fp32"), f"rank {r}: {first_mismatch(got, want[r])}"


def test_single_step_allgather_copy_inline():
    run_allgather(1, 5000, "bf16")
    with H.Comm(1, device=0) as c:
        x = inputs(1, 4097, "int32", 31)
        send = [to_device(x[0], "int32")]
        out = Guarded(4097, "int32")
        H.hccl_allgather(c.handle, send, [out.view], 4097, "int32")
        torch.cuda.synchronize()
        assert c.last_program()["inline_launch"] == 1
        assert np.array_equal(out.result(), x[0]) and out.guards_intact()


@pytest.mark.parametrize("rows_per_rank", [5000, 12000])
def test_group_of_embedding_rows_and_ids_is_one_launch(rows_per_rank):
    """5000 rows per rank cut every step into one 2048-element tile size; from about 8200 rows
    the bf16 row steps keep 4096-element tiles beside the int32 ids' 2048."""
    P = 8
    counts = zipf_counts(P, rows_per_rank, 1.1, seed=40)
    rows, ids = alltoallv_layout(counts, 128), alltoallv_layout(counts, 1)
    rng = np.random.default_rng(41)
    rows_h = [rng.integers(0, 2 ** 16, int(rows["send_len"][s]), dtype=np.int64).astype(np.uint16) for s in range(P)]
    ids_h = [rng.integers(-2 ** 31, 2 ** 31, int(ids["send_len"][s]), dtype=np.int64).astype(np.int32) for s in range(P)]
    print(f"group: alltoallv rows + ids, {rows_per_rank} rows per rank", flush=True)
    with H.Comm(P, device=0) as c:
        sr = [to_device(rows_h[s], "bf16") for s in range(P)]
        si = [to_device(ids_h[s], "int32") for s in range(P)]
        rr = [Guarded(int(rows["recv_len"][d]), "bf16") for d in range(P)]
        ri = [Guarded(int(ids["recv_len"][d]), "int32") for d in range(P)]
        with c.group():
            c.alltoallv(sr, rows["sendcounts"], rows["sdispls"], [o.view for o in rr], rows["recvcounts"], rows["rdispls"])
            c.alltoallv(si, ids["sendcounts"], ids["sdispls"], [o.view for o in ri], ids["recvcounts"], ids["rdispls"])
        torch.cuda.synchronize()
        info = c.last_program()
        assert c.async_error() == 0
    assert info["collective"] == -1
    tiles = (2048, 2048) if rows_per_rank == 5000 else (2048, 4096)
    assert (info["step_tile_min"], info["step_tile_max"]) == tiles, info
    want_r = [np.zeros(o.n, np.uint16) for o in rr]
    want_i = [np.zeros(o.n, np.int32) for o in ri]
    oracle.alltoallv(rows_h, rows["sendcounts"], rows["sdispls"], want_r, rows["recvcounts"], rows["rdispls"])
    oracle.alltoallv(ids_h, ids["sendcounts"], ids["sdispls"], want_i, ids["recvcounts"], ids["rdispls"])
    for d in range(P):
        assert np.array_equal(rr[d].result(), want_r[d]) and rr[d].guards_intact(), f"rows {d}"
        assert np.array_equal(ri[d].result(), want_i[d]) and ri[d].guards_intact(), f"ids {d}"


@pytest.mark.parametrize("fuse", [0, 1])
def test_group_of_dependent_programs_with_scratch(fuse):
    # two unfused ring collectives with FP32 scratch partials and dependency chains in one launch
    P = 4
    xa = inputs(P, 20000, "bf16", 42)
    xb = inputs(P, P * 3001, "bf16", 43)
    xc = inputs(P, 777, "fp32", 44)
    print(f"group: allreduce + reduce_scatter + allgather, fuse={fuse}", flush=True)
    with H.Comm(P, device=0, algo="ring", fuse=fuse, chunk_bytes=4096, tile_bytes=4096) as c:
        sa = [to_device(xa[r], "bf16") for r in range(P)]
        sb = [to_device(xb[r], "bf16") for r in range(P)]
        sc = [to_device(xc[r], "fp32") for r in range(P)]
        oa = [Guarded(20000, "bf16") for _ in range(P)]
        ob = [Guarded(3001, "bf16") for _ in range(P)]
        oc = [Guarded(P * 777, "fp32") for _ in range(P)]
        for _ in range(3):
            with c.group():
                c.allreduce(sa, [o.view for o in oa])
                c.reduce_scatter(sb, [o.view for o in ob])
                c.allgather(sc, [o.view for o in oc])
            torch.cuda.synchronize()
            assert c.async_error() == 0
    wa, wb, wc = oracle.allreduce(xa, "bf16"), oracle.reduce_scatter(xb, "bf16"), oracle.allgather(xc)
    for r in range(P):
        assert same_bits(oa[r].result(), wa[r], "bf16") and oa[r].guards_intact()
        assert same_bits(ob[r].result(), wb[r], "bf16") and ob[r].guards_intact()
        assert np.array_equal(oc[r].result().view(np.uint8), wc[r].view(np.uint8)) and oc[r].guards_intact()


@pytest.mark.parametrize("dt", ["bf16", "fp32"])
@pytest.mark.parametrize("algo", ["direct", "ring"])
@pytest.mark.parametrize("coll", ["reduce_scatter", "allreduce"])
def test_reduction_every_source_and_receive_alignment(dt, algo, coll):
    """Reductions of 4 ranks whose send and receive buffers start at every offset modulo 16, at
    one offset for every rank or at offsets that differ by rank (a reduce-scatter block's sources
    then agree with each other but not with the output, or disagree too); counts around the
    16-byte and wavefront boundaries. Bit-exact against the oracle's ascending fold."""
    es = DT_ES[dt]
    per = 16 // es
    P = 4
    print(f"reduction alignments {coll} dt={dt} algo={algo}", flush=True)
    with H.Comm(P, device=0, algo=algo, tile_bytes=2048) as c:
        for k, n in enumerate([1, per - 1, per + 1, 64 * per + 3, 131 * per + 5]):
            n_in = P * n if coll == "reduce_scatter" else n
            x = inputs(P, n_in, dt, seed=100 + k)
            want = oracle.reduce_scatter(x, dt) if coll == "reduce_scatter" else oracle.allreduce(x, dt)
            for so in range(per):
                for ro in range(per):
                    for mixed in (False, True):
                        soff = [(so + (r if mixed else 0)) % per for r in range(P)]
                        roff = [(ro + (2 * r if mixed else 0)) % per for r in range(P)]
                        send = [to_device(np.concatenate([np.zeros(soff[r], x.dtype), x[r]]), dt)[soff[r]:]
                                for r in range(P)]
                        outs = [Guarded(roff[r] + n + per, dt) for r in range(P)]
                        views = [o.view[roff[r]:roff[r] + n] for r, o in enumerate(outs)]
                        if coll == "reduce_scatter":
                            H.hccl_reduce_scatter(c.handle, send, views, n, dt)
                        else:
                            H.hccl_allreduce(c.handle, send, views, n, dt)
                        torch.cuda.synchronize()
                        for r in range(P):
                            got = outs[r].result()
                            where = (n, so, ro, mixed, r)
                            assert same_bits(got[roff[r]:roff[r] + n], want[r], dt), \
                                f"{where}: {first_mismatch(got[roff[r]:roff[r] + n], want[r])}"
                            init = outs[r].host_init[GUARD:GUARD + outs[r].n]
                            assert np.array_equal(got[:roff[r]].view(np.uint8), init[:roff[r]].view(np.uint8)), where
                            assert np.array_equal(got[roff[r] + n:].view(np.uint8), init[roff[r] + n:].view(np.uint8)), where
                            assert outs[r].guards_intact(), where
        assert c.async_error() == 0


@pytest.mark.parametrize("case", [
    ("reduce_scatter", "fp16", "max", dict(algo="direct"), "ascending", 0),
    ("reduce_scatter", "int32", "sum", dict(algo="ring"), "ascending", 0),
    ("reduce_scatter", "bf16", "min", dict(algo="ring"), "ascending", 0),
    ("reduce_scatter", "bf16", "sum", dict(algo="ring", fuse=0, requantize=1), "ascending", 0),
    ("allreduce", "bf16", "sum", dict(algo="two_level", group_size=2), "two_level", 2),
    ("allreduce", "fp16", "sum", dict(algo="two_level", group_size=2, fuse=0, requantize=1), "two_level", 2),
    ("allreduce", "fp32", "sum", dict(algo="two_level", group_size=2, fuse=0), "two_level", 2),
    ("reduce_scatter", "bf16", "sum", dict(algo="rhd", order="halving"), "halving", 0),
    ("allreduce", "fp32", "max", dict(algo="direct", order="halving"), "halving", 0),
    ("allreduce", "fp16", "sum", dict(algo="rhd", order="halving", fuse=0, requantize=1), "halving", 0),
], ids=lambda c: f"{c[0]}-{c[1]}-{c[2]}-{'-'.join(f'{k}{v}' for k, v in c[3].items())}")
def test_reduction_variants_at_shifted_offsets(case):
    """Grouped, re-quantised, unfused, MAX / MIN, fp16 and int32 reductions of 4 ranks with send
    and receive buffers at offsets modulo 16 that differ by rank and from each other, counts
    around the 16-byte and wavefront boundaries; against the oracle in the schedule's order."""
    coll, dt, op, cfg, order, group = case
    es = DT_ES[dt]
    per = 16 // es
    P = 4
    requant = bool(cfg.get("requantize", 0))
    print(f"shifted reductions {case}", flush=True)
    with H.Comm(P, device=0, tile_bytes=2048, chunk_bytes=4096, **cfg) as c:
        for k, n in enumerate([1, per + 1, 64 * per + 3, 131 * per + 5, 1500]):
            n_in = P * n if coll == "reduce_scatter" else n
            x = inputs(P, n_in, dt, seed=200 + k)
            if coll == "reduce_scatter":
                want = oracle.reduce_scatter_ordered(x, dt, order=order, op=op, group=group, requant=requant)
            else:
                want = oracle.allreduce_ordered(x, dt, order=order, op=op, group=group, requant=requant)
            for so, ro in [(0, 1), (1, 0), (per - 1, 2), (3 % per, per - 1)]:
                soff = [(so + r) % per for r in range(P)]
                roff = [(ro + 3 * r) % per for r in range(P)]
                send = [to_device(np.concatenate([np.zeros(soff[r], x.dtype), x[r]]), dt)[soff[r]:] for r in range(P)]
                outs = [Guarded(roff[r] + n + per, dt) for r in range(P)]
                views = [o.view[roff[r]:roff[r] + n] for r, o in enumerate(outs)]
                if coll == "reduce_scatter":
                    H.hccl_reduce_scatter(c.handle, send, views, n, dt, op)
                else:
                    H.hccl_allreduce(c.handle, send, views, n, dt, op)
                torch.cuda.synchronize()
                for r in range(P):
                    got = outs[r].result()
                    where = (n, so, ro, r)
                    assert same_bits(got[roff[r]:roff[r] + n], want[r], dt), \
                        f"{where}: {first_mismatch(got[roff[r]:roff[r] + n], want[r])}"
                    init = outs[r].host_init[GUARD:GUARD + outs[r].n]
                    assert np.array_equal(got[:roff[r]].view(np.uint8), init[:roff[r]].view(np.uint8)), where
                    assert np.array_equal(got[roff[r] + n:].view(np.uint8), init[roff[r] + n:].view(np.uint8)), where
                    assert outs[r].guards_intact(), where
        assert c.async_error() == 0


@pytest.mark.parametrize("es_dt", ["bf16", "int32"])
@pytest.mark.parametrize("algo", ["direct", "ring"])
def test_allgather_every_source_and_receive_alignment(es_dt, algo):
    """All-gathers of 4 ranks whose send blocks start at every offset modulo 16 and whose blocks
    land at every offset modulo 16: every rank's receive buffer at the same offset (the
    destinations of a direct copy agree among themselves but not with the source) or at offsets
    that differ by rank; counts around the 16-byte and wavefront boundaries."""
    es = 2 if es_dt == "bf16" else 4
    per = 16 // es
    P = 4
    rng = np.random.default_rng(40 + es)
    print(f"allgather alignments dt={es_dt} algo={algo}", flush=True)
    with H.Comm(P, device=0, algo=algo, tile_bytes=2048) as c:
        for n in [1, per - 1, per + 1, 64 * per + 3, 131 * per + 5]:
            for so in range(per):
                for ro in range(per):
                    for mixed in (False, True):
                        roff = [(ro + (r if mixed else 0)) % per for r in range(P)]
                        src = [rng.integers(0, 1 << 15, size=so + n).astype(np.uint16 if es == 2 else np.int32)
                               for _ in range(P)]
                        send = [to_device(x, es_dt)[so:] for x in src]
                        outs = [Guarded(roff[r] + P * n + per, es_dt) for r in range(P)]
                        H.hccl_allgather(c.handle, send, [o.view[roff[r]:roff[r] + P * n] for r, o in enumerate(outs)],
                                         n, es_dt)
                        torch.cuda.synchronize()
                        gathered = oracle.allgather(np.stack([x[so:] for x in src]))
                        for r in range(P):
                            want = outs[r].host_init[GUARD:GUARD + outs[r].n].copy()
                            want[roff[r]:roff[r] + P * n] = gathered[r]
                            got = outs[r].result()
                            assert np.array_equal(got.view(np.uint8), want.view(np.uint8)), (n, so, ro, mixed, r)
                            assert outs[r].guards_intact(), (n, so, ro, mixed, r)
        assert c.async_error() == 0


@pytest.mark.parametrize("es_dt", ["bf16", "int32"])
def test_copy_every_source_and_destination_alignment(es_dt):
    """Every (source, destination) byte offset modulo 16 and lengths around the 16-byte and
    wavefront boundaries, as one-rank AllToAllv copies (the offsets set the alignments)."""
    es = 2 if es_dt == "bf16" else 4
    per = 16 // es
    lengths = [1, 2, per - 1, per, per + 1, 3 * per + 1, 64 * per - 1, 64 * per, 64 * per + 3, 131 * per + 5,
               1000]
    print(f"copy alignments dt={es_dt}", flush=True)
    rng = np.random.default_rng(es)
    with H.Comm(1, device=0, tile_bytes=2048) as c:
        for n in lengths:
            for so in range(per):
                for ro in range(per):
                    src = rng.integers(0, 1 << 15, size=so + n + per).astype(np.uint16 if es == 2 else np.int32)
                    send = to_device(src, es_dt)
                    out = Guarded(ro + n + per, es_dt)
                    H.hccl_alltoallv(c.handle, [send], [n], [so], [out.view], [n], [ro], es_dt)
                    torch.cuda.synchronize()
                    got = out.result()
                    want = out.host_init[GUARD:GUARD + ro + n + per].copy()
                    want[ro:ro + n] = src[so:so + n]
                    assert np.array_equal(got.view(np.uint8), want.view(np.uint8)), (n, so, ro)
                    assert out.guards_intact(), (n, so, ro)
        assert c.async_error() == 0
