"""Host logic: lowering, fusion, packing and validation of descriptor programs.

These run on host-only communicators (device = HCCL_NO_DEVICE): a collective call checks its
arguments, compiles the program and runs the validator (dependency order, bounds, races under
the dependency closure, scratch read-after-write, exact output coverage), then returns
without touching memory. No GPU is needed.
"""
import numpy as np
import pytest

import paper_2608_00358_amd as H
from workloads import alltoallv_layout, zipf_counts

ES = {"bf16": 2, "fp16": 2, "fp32": 4, "int32": 4}
GiB = 1 << 30


def fake_bufs(P, base):
    # distinct, 4 KiB aligned, far apart: never dereferenced on a host-only communicator
    return [base + i * (1 << 36) for i in range(P)]


def comm(P, **cfg):
    return H.Comm(P, device=H.NO_DEVICE, **cfg)


def info_of(c):
    return c.last_program()


def ceil_div(a, b):
    return -(-a // b)


@pytest.mark.parametrize("dt", ["bf16", "fp32", "int32", "fp16"])
@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("fuse", [0, 1])
def test_reduce_scatter_ring_structure(dt, P, fuse):
    M = 3 * 4096 + 17
    chunk = 8192
    with comm(P, algo="ring", fuse=fuse, chunk_bytes=chunk) as c:
        H.hccl_reduce_scatter(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), M, dt)
        info = info_of(c)
    C = chunk // ES[dt]
    chains = P * ceil_div(M, C)
    if fuse or P <= 2:
        assert info["num_descs"] == chains * (1 if P <= 2 or fuse else P - 1)
    else:
        assert info["num_descs"] == chains * (P - 1)
    if fuse:
        assert info["num_deps"] == 0 and info["max_srcs"] == P
        assert info["bytes_read"] == P * P * M * ES[dt]
        assert info["bytes_written"] == P * M * ES[dt]
        assert info["scratch_bytes"] == 0


@pytest.mark.parametrize("algo", ["direct", "ring"])
@pytest.mark.parametrize("P", [1, 2, 4, 5])
@pytest.mark.parametrize("fuse", [0, 1])
@pytest.mark.parametrize("phases", ["auto", "one"])
def test_allreduce_structure_and_minimal_traffic_when_fused(algo, P, fuse, phases):
    N = 100003
    dt = "bf16"
    with comm(P, algo=algo, fuse=fuse, chunk_bytes=65536, phases=phases) as c:
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), N, dt)
        info = info_of(c)
    if fuse or algo == "direct":
        assert info["num_deps"] == 0 and info["num_phases"] == 1
        assert info["bytes_read"] == P * N * 2 and info["bytes_written"] == P * N * 2
    elif P > 1:
        assert info["bytes_read"] > P * N * 2
        if phases == "one":
            # one launch: the ring's hops wait for each other tile by tile on the device
            assert info["num_deps"] > 0 and info["num_phases"] == 1
        else:
            # one launch per hop: P-2 reduce hops after the first, P-1 forwarding hops
            assert info["num_deps"] == 0 and info["num_phases"] == max(1, P - 1) + (P - 1)


def test_allreduce_in_place_is_validated_with_aliasing():
    P, N = 4, 50000
    bufs = fake_bufs(P, 1 << 40)
    for fuse in (0, 1):
        with comm(P, algo="ring", fuse=fuse, chunk_bytes=16384) as c:
            H.hccl_allreduce(c.handle, bufs, bufs, N, "fp32")


@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("fuse", [0, 1])
def test_allgather_ring_fuses_to_one_copy_per_chunk(P, fuse):
    M = 70001
    with comm(P, algo="ring", fuse=fuse, chunk_bytes=65536) as c:
        H.hccl_allgather(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), M, "bf16")
        info = info_of(c)
    chunks = ceil_div(M, 65536 // 2)
    if fuse:
        assert info["num_descs"] == P * chunks and info["num_deps"] == 0
        assert info["bytes_read"] == P * M * 2 and info["bytes_written"] == P * P * M * 2
    else:
        assert info["num_descs"] == P * P * chunks


@pytest.mark.parametrize("L,G", [(8, 8), (2, 4), (4, 2), (1, 4), (4, 1)])
@pytest.mark.parametrize("fuse", [0, 1])
def test_two_level_structure(L, G, fuse):
    P = L * G
    N = 1 << 16
    with comm(P, algo="two_level", group_size=L, fuse=fuse, chunk_bytes=16384) as c:
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), N, "bf16")
        info = info_of(c)
    assert info["algo"] == 3
    if fuse:
        assert info["num_deps"] == 0 and info["scratch_bytes"] == 0
        assert info["bytes_read"] == P * N * 2 and info["bytes_written"] == P * N * 2
        assert info["max_srcs"] == P
    else:
        assert info["scratch_bytes"] == G * N * 4


def test_auto_picks_two_level_when_group_size_splits_ranks():
    with comm(16, group_size=4) as c:
        H.hccl_allreduce(c.handle, fake_bufs(16, 1 << 40), fake_bufs(16, 1 << 44), 4096, "bf16")
        assert info_of(c)["algo"] == 3
    with comm(16, group_size=5) as c:
        H.hccl_allreduce(c.handle, fake_bufs(16, 1 << 40), fake_bufs(16, 1 << 44), 4096, "bf16")
        assert info_of(c)["algo"] == 2


def test_alltoallv_zipf_layout_compiles_and_counts_bytes():
    P, R, D = 8, 1 << 12, 128
    counts = zipf_counts(P, R, 1.1, seed=0)
    lay = alltoallv_layout(counts, D)
    chunk = 1 << 16
    with comm(P, chunk_bytes=chunk) as c:
        H.hccl_alltoallv(c.handle, fake_bufs(P, 1 << 40), lay["sendcounts"], lay["sdispls"],
                         fake_bufs(P, 1 << 44), lay["recvcounts"], lay["rdispls"], "bf16")
        info = info_of(c)
    total = int(lay["sendcounts"].sum()) * 2
    assert info["bytes_read"] == total and info["bytes_written"] == total
    pieces = sum(ceil_div(int(n) * 2, chunk) for n in lay["sendcounts"].reshape(-1) if n)
    assert info["num_descs"] == pieces


def test_program_cache_reuses_compiled_programs():
    with comm(4) as c:
        s, r = fake_bufs(4, 1 << 40), fake_bufs(4, 1 << 44)
        H.hccl_allreduce(c.handle, s, r, 1000, "fp32")
        assert info_of(c)["cache_hit"] == 0
        H.hccl_allreduce(c.handle, fake_bufs(4, 1 << 41), fake_bufs(4, 1 << 45), 1000, "fp32")
        assert info_of(c)["cache_hit"] == 1       # other buffers, same shape: cached
        H.hccl_allreduce(c.handle, s, r, 1001, "fp32")
        assert info_of(c)["cache_hit"] == 0


# ----------------------------------------------------------------------- error paths
def _expect(code, fn, *args):
    with pytest.raises(H.HcclError) as e:
        fn(*args)
    assert e.value.code == code, str(e.value)


def test_rejects_overlapping_buffers_and_partial_in_place():
    P = 4
    with comm(P) as c:
        s = fake_bufs(P, 1 << 40)
        r = list(s)
        r[1] = s[1] + 8
        _expect(1, H.hccl_allreduce, c.handle, s, r, 1000, "fp32")
        r2 = fake_bufs(P, 1 << 44)
        r2[2] = s[2]
        _expect(1, H.hccl_allreduce, c.handle, s, r2, 1000, "fp32")
        _expect(1, H.hccl_reduce_scatter, c.handle, s, s, 1000, "fp32")


def test_rejects_misaligned_and_null_buffers():
    P = 2
    with comm(P) as c:
        s, r = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
        s[0] += 2
        _expect(1, H.hccl_allreduce, c.handle, s, r, 100, "fp32")
        s, r = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
        r[1] = 0
        _expect(1, H.hccl_allreduce, c.handle, s, r, 100, "fp32")


def test_rejects_bad_enums():
    with comm(2) as c:
        s, r = fake_bufs(2, 1 << 40), fake_bufs(2, 1 << 44)
        _expect(1, H.hccl_allreduce, c.handle, s, r, 100, 7)


def test_alltoallv_rejects_inconsistent_counts_and_overlapping_receive_ranges():
    P = 3
    counts = np.array([[1, 2, 3], [4, 5, 6], [7, 8, 9]])
    lay = alltoallv_layout(counts)
    with comm(P) as c:
        s, r = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
        bad = lay["recvcounts"].copy()
        bad[0, 2] += 1
        _expect(1, H.hccl_alltoallv, c.handle, s, lay["sendcounts"], lay["sdispls"], r, bad, lay["rdispls"], "fp32")
        rd = lay["rdispls"].copy()
        rd[1, 1] = rd[1, 0]
        _expect(1, H.hccl_alltoallv, c.handle, s, lay["sendcounts"], lay["sdispls"], r, lay["recvcounts"], rd, "fp32")


def test_two_level_rejected_for_reduce_scatter():
    with comm(4, algo="two_level", group_size=2) as c:
        _expect(2, H.hccl_reduce_scatter, c.handle, fake_bufs(4, 1 << 40), fake_bufs(4, 1 << 44), 10, "fp32")


def test_empty_collectives_compile_to_nothing():
    with comm(4) as c:
        H.hccl_allreduce(c.handle, fake_bufs(4, 1 << 40), fake_bufs(4, 1 << 44), 0, "bf16")
        assert info_of(c)["num_tiles"] == 0
        z = np.zeros((4, 4), dtype=np.int64)
        H.hccl_alltoallv(c.handle, fake_bufs(4, 1 << 40), z, z, fake_bufs(4, 1 << 44), z, z, "bf16")
        assert info_of(c)["num_tiles"] == 0


# -------------------------------------------------------------------------- groups
def test_group_merges_calls_into_one_program():
    P = 4
    with comm(P, algo="ring", fuse=0, chunk_bytes=4096) as c:
        s1, r1 = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
        H.hccl_allreduce(c.handle, s1, r1, 5000, "bf16")
        one = info_of(c)
        s2, r2 = fake_bufs(P, 1 << 42), fake_bufs(P, 1 << 46)
        H.hccl_reduce_scatter(c.handle, s2, r2, 3000, "fp32")
        two = info_of(c)
        H.hccl_group_start(c.handle)
        H.hccl_allreduce(c.handle, s1, r1, 5000, "bf16")
        H.hccl_reduce_scatter(c.handle, s2, r2, 3000, "fp32")
        H.hccl_group_end(c.handle)
        g = info_of(c)
    assert g["num_descs"] == one["num_descs"] + two["num_descs"]
    assert g["num_deps"] == one["num_deps"] + two["num_deps"]
    assert g["bytes_read"] == one["bytes_read"] + two["bytes_read"]
    assert g["scratch_bytes"] >= one["scratch_bytes"] + two["scratch_bytes"]
    assert g["collective"] == -1


@pytest.mark.parametrize("rows_per_rank, tiles", [(5000, (2048, 2048)), (12000, (2048, 4096)),
                                                  (1 << 18, (2048, 4096))])
def test_grouped_rows_and_ids_tile_each_step_by_its_width(rows_per_rank, tiles):
    """The embedding exchange recorded as one group (rows of 128 bf16 plus int32 ids): without
    dependencies every step is cut by its own element width (8 KiB tiles: 4096 bf16 or 2048
    int32 elements), capped so that small programs still spread over 2048 tiles."""
    P, D = 8, 128
    counts = zipf_counts(P, rows_per_rank, 1.1, seed=0)
    rows, ids = alltoallv_layout(counts, D), alltoallv_layout(counts, 1)
    with comm(P) as c:
        H.hccl_group_start(c.handle)
        H.hccl_alltoallv(c.handle, fake_bufs(P, 1 << 40), rows["sendcounts"], rows["sdispls"], fake_bufs(P, 1 << 44),
                         rows["recvcounts"], rows["rdispls"], "bf16")
        H.hccl_alltoallv(c.handle, fake_bufs(P, 1 << 42), ids["sendcounts"], ids["sdispls"], fake_bufs(P, 1 << 46),
                         ids["recvcounts"], ids["rdispls"], "int32")
        H.hccl_group_end(c.handle)
        info = info_of(c)
    assert (info["step_tile_min"], info["step_tile_max"]) == tiles
    payload = int(rows["sendcounts"].sum()) * 2 + int(ids["sendcounts"].sum()) * 4
    assert info["bytes_read"] == info["bytes_written"] == payload
    assert info["num_deps"] == 0 and info["scratch_bytes"] == 0


def test_group_rejects_overlap_between_calls_and_unbalanced_end():
    P = 2
    with comm(P) as c:
        s, r = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
        H.hccl_group_start(c.handle)
        H.hccl_allreduce(c.handle, s, r, 100, "fp32")
        H.hccl_allreduce(c.handle, r, fake_bufs(P, 1 << 42), 100, "fp32")   # reads what the first writes
        _expect(1, H.hccl_group_end, c.handle)
        _expect(1, H.hccl_group_end, c.handle)


def test_group_rejects_too_many_buffers_and_nests():
    with comm(64) as c:
        H.hccl_group_start(c.handle)
        H.hccl_group_start(c.handle)      # nested: only the outer end launches
        for k in range(2):
            H.hccl_allgather(c.handle, fake_bufs(64, (1 << 40) + k * (1 << 35)),
                             fake_bufs(64, (1 << 44) + k * (1 << 35)), 10, "bf16")
        H.hccl_group_end(c.handle)
        _expect(2, H.hccl_group_end, c.handle)   # 2 x 128 rank buffers > 128


def test_empty_group_is_a_no_op():
    with comm(2) as c:
        H.hccl_group_start(c.handle)
        H.hccl_group_end(c.handle)


# ------------------------------------------------------------- fold orders and RHD
@pytest.mark.parametrize("P", [1, 2, 4, 8])
@pytest.mark.parametrize("fuse", [0, 1])
def test_rhd_reduce_scatter_structure(P, fuse):
    M, chunk = 5000, 4096
    with comm(P, algo="rhd", order="halving", fuse=fuse, chunk_bytes=chunk, phases="one") as c:
        H.hccl_reduce_scatter(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), M, "bf16")
        info = info_of(c)
    chunks = ceil_div(M, chunk // 2)
    assert info["algo"] == 4
    if fuse or P == 1:
        # every butterfly level merged: one binary-tree step per block chunk, minimal traffic
        assert info["num_descs"] == P * chunks and info["num_deps"] == 0
        assert info["max_srcs"] == P and info["scratch_bytes"] == 0
        assert info["bytes_read"] == P * P * M * 2
    else:
        # P ranks x (P-1) kept blocks summed over the levels, per chunk
        assert info["num_descs"] == P * (P - 1) * chunks
        assert (info["num_deps"] > 0) == (P > 2)     # one level has nothing to wait for
        assert info["num_phases"] == 1
    # by default the butterfly levels are launches of their own and wait for nothing on the device
    with comm(P, algo="rhd", order="halving", fuse=fuse, chunk_bytes=chunk) as c:
        H.hccl_reduce_scatter(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), M, "bf16")
        auto = info_of(c)
    assert auto["num_deps"] == 0 and auto["num_descs"] == info["num_descs"]
    assert auto["num_phases"] == (1 if fuse or P == 1 else P.bit_length() - 1)


@pytest.mark.parametrize("P", [2, 4, 8])
@pytest.mark.parametrize("fuse", [0, 1])
def test_rhd_allreduce_and_allgather_validate(P, fuse):
    with comm(P, algo="rhd", order="halving", fuse=fuse, chunk_bytes=4096) as c:
        s, r = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
        H.hccl_allreduce(c.handle, s, r, 20001, "fp32")
        ar = info_of(c)
        H.hccl_allreduce(c.handle, s, s, 20001, "fp32")          # in place, aliasing checked
        H.hccl_allgather(c.handle, s, r, 3001, "bf16")
        ag = info_of(c)
    if fuse:
        assert ar["num_deps"] == 0 and ar["bytes_written"] == P * 20001 * 4
        assert ag["num_deps"] == 0 and ag["bytes_read"] == P * 3001 * 2


@pytest.mark.parametrize("order", ["ring", "halving"])
def test_direct_schedule_takes_any_order(order):
    P = 8
    with comm(P, algo="direct", order=order) as c:
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), 100000, "bf16")
        info = info_of(c)
    if order == "ring":
        assert info["num_descs"] == P          # one step per shard: each has its own rotation
    else:
        assert info["num_descs"] == 1


def test_requantized_partials_are_stored_in_the_buffer_type():
    P, N = 4, 1 << 14
    for requant, width in ((0, 4), (1, 2)):
        with comm(P, algo="ring", fuse=0, requantize=requant) as c:
            H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), N, "bf16")
            assert info_of(c)["scratch_bytes"] == N * width


def test_incompatible_orders_and_schedules_are_rejected():
    s, r = fake_bufs(6, 1 << 40), fake_bufs(6, 1 << 44)
    with comm(6, order="halving") as c:
        _expect(2, H.hccl_allreduce, c.handle, s, r, 100, "fp32")      # not a power of two
    with comm(4, algo="ring", order="halving") as c:
        _expect(2, H.hccl_allreduce, c.handle, s[:4], r[:4], 100, "fp32")
    with comm(4, algo="rhd") as c:
        _expect(2, H.hccl_allreduce, c.handle, s[:4], r[:4], 100, "fp32")
    with comm(4, algo="two_level", group_size=2, order="ring") as c:
        _expect(2, H.hccl_allreduce, c.handle, s[:4], r[:4], 100, "fp32")
    with comm(4, order=7) as c:
        _expect(1, H.hccl_allreduce, c.handle, s[:4], r[:4], 100, "fp32")


# ------------------------------------------------------------------ AllToAllvDynamic
def dyn_slots(P, send_cap, R, es, tile_bytes=8192):
    te = max(512, (tile_bytes // es) // 512 * 512)
    bound = P * (ceil_div(send_cap * R, te) + P)
    return max(1, min(32768, bound))


META = 1 << 47   # fake device metadata arrays, far from the data buffers


@pytest.mark.parametrize("P", [1, 2, 8, 64])
@pytest.mark.parametrize("dt", ["bf16", "int32"])
def test_dynamic_alltoallv_is_a_plan_and_a_copy(P, dt):
    R, send_cap, recv_cap = 128, 5000, 7000
    with comm(P) as c:
        H.hccl_alltoallv_dynamic(c.handle, fake_bufs(P, 1 << 40), META, None, fake_bufs(P, 1 << 44), None, None,
                                 R, send_cap, recv_cap, dt)
        info = info_of(c)
        # one step of slots, each planning the whole exchange itself: no dependencies, no scratch
        assert info["collective"] == 4 and info["num_descs"] == 1 and info["num_deps"] == 0
        assert info["num_tiles"] == dyn_slots(P, send_cap, R, ES[dt])
        assert info["scratch_bytes"] == 0 and info["num_operands"] == 0
        # the program does not depend on the counts: other metadata arrays reuse it
        H.hccl_alltoallv_dynamic(c.handle, fake_bufs(P, 1 << 40), META + (1 << 20), META + (2 << 20),
                                 fake_bufs(P, 1 << 44), META + (3 << 20), None, R, send_cap, recv_cap, dt)
        assert info_of(c)["cache_hit"] == 0    # explicit send offsets and a count output: another program
        H.hccl_alltoallv_dynamic(c.handle, fake_bufs(P, 1 << 41), META + (5 << 20), META + (6 << 20),
                                 fake_bufs(P, 1 << 45), META + (7 << 20), None, R, send_cap, recv_cap, dt)
        assert info_of(c)["cache_hit"] == 1


def test_dynamic_alltoallv_small_capacities_get_few_slots():
    with comm(2) as c:
        H.hccl_alltoallv_dynamic(c.handle, fake_bufs(2, 1 << 40), META, None, fake_bufs(2, 1 << 44), None, None,
                                 1, 3, 6, "fp32")
        assert info_of(c)["num_tiles"] == 2 * (1 + 2)
        H.hccl_alltoallv_dynamic(c.handle, fake_bufs(2, 1 << 40), META, None, fake_bufs(2, 1 << 44), None, None,
                                 1, 0, 0, "fp32")
        assert info_of(c)["num_tiles"] == 2 * 2


def test_dynamic_alltoallv_argument_errors():
    P = 4
    s, r = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
    with comm(P) as c:
        f = H.hccl_alltoallv_dynamic
        _expect(1, f, c.handle, s, None, None, r, None, None, 8, 10, 10, "bf16")          # no counts
        _expect(1, f, c.handle, s, META, None, r, None, None, 0, 10, 10, "bf16")          # row_elems 0
        _expect(1, f, c.handle, s, META + 4, None, r, None, None, 8, 10, 10, "bf16")      # misaligned
        _expect(1, f, c.handle, s, META, None, r, None, None, 8, 1 << 60, 10, "bf16")     # capacity
        _expect(1, f, c.handle, s, META, None, r, r[1], None, 8, 10, 10, "bf16")          # output on a receive
        _expect(1, f, c.handle, s, META, None, r, META + 64, None, 8, 10, 10, "bf16")     # output on the counts
        _expect(1, f, c.handle, s, META, None, r, None, r[2] + 8, 8, 10, 10, "bf16")      # offsets on a receive
        f(c.handle, s, s[0], s[1], r, None, None, 8, 10, 10, "bf16")                        # read-only aliases
        _expect(2, f, c.handle, s, META, None, r, None, None, 1 << 20, 1 << 21, 10, "bf16")  # too many tiles


def test_dynamic_alltoallv_groups():
    P = 8
    with comm(P) as c:
        # embedding rows and their ids exchanged with one count matrix: two dynamic calls
        with c.group():
            H.hccl_alltoallv_dynamic(c.handle, fake_bufs(P, 1 << 40), META, None, fake_bufs(P, 1 << 44), None,
                                     None, 128, 4096, 4096, "bf16")
            H.hccl_alltoallv_dynamic(c.handle, fake_bufs(P, 1 << 41), META, None, fake_bufs(P, 1 << 45),
                                     META + (1 << 20), None, 1, 4096, 4096, "int32")
            H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 42), fake_bufs(P, 1 << 43), 1000, "fp32")
        g = info_of(c)
        assert g["collective"] == -1 and g["num_deps"] == 0 and g["num_descs"] >= 3
        H.hccl_group_start(c.handle)
        for k in range(3):
            H.hccl_alltoallv_dynamic(c.handle, fake_bufs(P, (1 << 40) + k * (1 << 37)), META, None,
                                     fake_bufs(P, (1 << 44) + k * (1 << 37)), None, None, 1, 64, 64, "fp32")
        _expect(2, H.hccl_group_end, c.handle)
        # two calls writing the same count output conflict
        H.hccl_group_start(c.handle)
        for k in range(2):
            H.hccl_alltoallv_dynamic(c.handle, fake_bufs(P, (1 << 40) + k * (1 << 37)), META, None,
                                     fake_bufs(P, (1 << 44) + k * (1 << 37)), META + (1 << 20), None, 1, 64, 64,
                                     "fp32")
        _expect(1, H.hccl_group_end, c.handle)


# ------------------------------------------------------------------------- triggers
def test_trigger_arguments_and_consumption():
    P = 4
    s, r = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
    word = META
    with comm(P) as c:
        _expect(1, H.hccl_set_trigger, c.handle, (word + 4, "eq", 1), None)            # misaligned
        _expect(1, H.hccl_set_trigger, c.handle, (word, "eq", 1), (word, 2))           # same word
        _expect(1, H.hccl_set_trigger, c.handle, (word, 9, 1), None)                   # comparator
        # a word inside a receive buffer is rejected when the packet is enqueued ...
        H.hccl_set_trigger(c.handle, (r[1] + 64, "ge", 1), None)
        _expect(1, H.hccl_allreduce, c.handle, s, r, 100, "fp32")
        # ... and the trigger went with that packet: the next call is untriggered
        H.hccl_allreduce(c.handle, s, r, 100, "fp32")
        # an empty packet cannot carry a trigger
        H.hccl_set_trigger(c.handle, None, (word, 1))
        _expect(1, H.hccl_allreduce, c.handle, s, r, 0, "fp32")
        H.hccl_set_trigger(c.handle, (word, "lt", 3), (word + 8, 1))
        H.hccl_set_trigger(c.handle)                                                    # cleared
        H.hccl_allreduce(c.handle, s, r, 0, "fp32")


# ------------------------------------------------------------------ environment overrides
def test_hccl_algo_and_chunk_bytes_override_the_configuration(monkeypatch):
    P, N = 4, 40000
    monkeypatch.setenv("HCCL_ALGO", "direct")
    monkeypatch.setenv("HCCL_CHUNK_BYTES", "16K")
    with comm(P, algo="ring", chunk_bytes=1 << 20) as c:
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), N, "fp32")
        info = info_of(c)
    assert info["algo"] == 1                               # direct, not the configured ring
    assert info["num_descs"] == ceil_div(N, 16384 // 4)    # one step per 16 KiB chunk
    monkeypatch.setenv("HCCL_ALGO", "no-such-schedule")
    monkeypatch.delenv("HCCL_CHUNK_BYTES")
    with comm(P, algo="ring", fuse=0) as c:              # an unknown value is ignored
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), N, "fp32")
        assert info_of(c)["algo"] == 2


def test_hccl_debug_logs_creation_compiles_and_cache_hits(monkeypatch, capfd):
    monkeypatch.setenv("HCCL_DEBUG", "TRACE")
    with comm(2) as c:
        for _ in range(2):
            H.hccl_allgather(c.handle, fake_bufs(2, 1 << 40), fake_bufs(2, 1 << 44), 1000, "bf16")
    err = capfd.readouterr().err
    assert "[hccl INFO]" in err and "created: 2 ranks" in err
    assert "compiled allgather" in err and "[hccl TRACE]" in err and "cached program" in err
    monkeypatch.setenv("HCCL_DEBUG", "WARN")
    with comm(2) as c:
        H.hccl_allgather(c.handle, fake_bufs(2, 1 << 40), fake_bufs(2, 1 << 44), 1000, "bf16")
    assert capfd.readouterr().err == ""


# ------------------------------------------------------------------------------ phases
@pytest.mark.parametrize("kib,split", [(32 * 1024, True), (4 * 1024, True), (2 * 1024, False), (256, False)])
def test_wide_allreduce_splits_its_copies_only_when_large(kib, split):
    """The two-level all-reduce of 64 ranks: at 32 MiB per rank the 64-source reductions write
    one destination each and a second launch copies every result to the other 63 ranks (from 4 MiB
    per rank); at 2 MiB or 256 KiB per rank the fused one-launch program is kept."""
    P, N = 64, kib * 1024 // 2
    with comm(P, algo="two_level", group_size=8, validate=1) as c:
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), N, "bf16")
        info = info_of(c)
    assert info["num_deps"] == 0 and info["max_srcs"] == P
    if split:
        assert info["num_phases"] == 2
        assert info["bytes_read"] == (P + 1) * N * 2 and info["bytes_written"] == P * N * 2
        # the wide copies read up to 32 KiB per tile, in at least about 256 tiles
        assert info["step_tile_max"] == max(8192, min(32768, N * 2 // 256)) // 2
    else:
        assert info["num_phases"] == 1
        assert info["bytes_read"] == P * N * 2 and info["bytes_written"] == P * N * 2
    with comm(P, algo="two_level", group_size=8, phases="one") as c:
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), N, "bf16")
        assert info_of(c)["num_phases"] == 1 and info_of(c)["bytes_read"] == P * N * 2


@pytest.mark.parametrize("phases,launches", [("auto", 3), ("levels", 3), ("one", 1)])
def test_unfused_two_level_runs_level_by_level(phases, launches):
    """Unfused two-level schedule: group reductions, the reduction of the group partials, then
    the forwarding copies (the inter-group copy and the intra-group copies it feeds are merged
    by nothing, fusion being off: three dependency levels, plus one for copies of copies)."""
    P, N = 16, 100000
    with comm(P, algo="two_level", group_size=4, fuse=0, phases=phases, validate=1) as c:
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), N, "fp32")
        info = info_of(c)
    if phases == "one":
        assert info["num_phases"] == 1 and info["num_deps"] > 0
    else:
        assert info["num_phases"] == 4 and info["num_deps"] == 0


def test_phase_mode_is_part_of_the_cached_program():
    P, N = 4, 50000
    with comm(P, algo="ring", fuse=0) as c:
        s, r = fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44)
        H.hccl_allreduce(c.handle, s, r, N, "fp32")
        assert info_of(c)["num_phases"] > 1
        c.set_config(algo="ring", fuse=0, phases="one")
        H.hccl_allreduce(c.handle, s, r, N, "fp32")
        assert info_of(c)["num_phases"] == 1 and info_of(c)["cache_hit"] == 0
        with pytest.raises(H.HcclError):
            c.set_config(algo="ring", phases=7)
            H.hccl_allreduce(c.handle, s, r, N, "fp32")


@pytest.mark.parametrize("mib,tile_kib", [(1, 8), (4, 16), (8, 32), (32, 32)])
def test_wide_copies_keep_about_256_tiles(mib, tile_kib):
    """Forced split (phases=levels): the wide copies read the phase's copy bytes / 256 per tile,
    at least 8 KiB and at most 32 KiB."""
    P, N = 64, mib * (1 << 20) // 2
    with comm(P, algo="two_level", group_size=8, phases="levels") as c:
        H.hccl_allreduce(c.handle, fake_bufs(P, 1 << 40), fake_bufs(P, 1 << 44), N, "bf16")
        info = info_of(c)
    assert info["num_phases"] == 2 and info["step_tile_max"] == tile_kib * 1024 // 2
