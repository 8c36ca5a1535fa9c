"""Pins of the oracle's AllToAllvDynamic (paper Section IV-B-2, device-resident collectives).

The dynamic variant is an AllToAllv whose row counts (and optionally row offsets) are read
when it runs. These pins fix it against things outside its own code: a worked example whose
expected buffers are written out by hand, brute-force row placement in pure Python, the
plain AllToAllv oracle (itself pinned by brute force) fed with hand-computed element layouts,
and the layout rules (capacity, overlap, zero-count ranges) at their boundaries.
"""
import numpy as np
import pytest

import oracle

SENTINEL = -99


def rows_of(buf, row_elems):
    return buf.reshape(-1, row_elems)


def test_worked_example_packed_layout():
    # P = 2, rows of 2 int32 elements. Source 0 sends 1 row to rank 0 and 2 rows to rank 1;
    # source 1 sends nothing to rank 0 and 3 rows to rank 1.
    counts = np.array([[1, 2], [0, 3]])
    send0 = np.array([10, 11, 20, 21, 30, 31, 40, 41], np.int32)  # 4 rows of capacity
    send1 = np.array([50, 51, 60, 61, 70, 71, 80, 81], np.int32)
    recv = [np.full(10, SENTINEL, np.int32) for _ in range(2)]       # 5 rows of capacity
    ok, rcounts = oracle.alltoallv_dynamic([send0, send1], counts, recv, row_elems=2, send_cap=4, recv_cap=5)
    assert ok
    # rank 0 receives row 0 of source 0; rank 1 receives rows 1-2 of source 0 then rows 0-2 of source 1
    assert recv[0].tolist() == [10, 11] + [SENTINEL] * 8
    assert recv[1].tolist() == [20, 21, 30, 31, 50, 51, 60, 61, 70, 71]
    assert rcounts.tolist() == [[1, 0], [2, 3]]


def test_worked_example_explicit_offsets():
    counts = np.array([[1, 2], [0, 3]])
    send0 = np.array([10, 11, 20, 21, 30, 31, 40, 41], np.int32)
    send1 = np.array([50, 51, 60, 61, 70, 71, 80, 81], np.int32)
    # source 0's rows for rank 1 start at row 2, its row for rank 0 at row 0; source 1's at row 1
    sd = np.array([[0, 2], [3, 1]])           # sd[1, 0] is never read: that range is empty
    # rank 1 places source 1 first (row 0) and source 0 after a one-row gap (row 4)
    rd = np.array([[2, 99], [4, 0]])          # rd[0, 1] is never read: that range is empty
    recv = [np.full(12, SENTINEL, np.int32) for _ in range(2)]
    ok, _ = oracle.alltoallv_dynamic([send0, send1], counts, recv, row_elems=2, send_cap=4, recv_cap=6,
                                     sdispls=sd, rdispls=rd)
    assert ok
    assert recv[0].tolist() == [SENTINEL] * 4 + [10, 11] + [SENTINEL] * 6
    assert recv[1].tolist() == [60, 61, 70, 71, 80, 81, SENTINEL, SENTINEL, 30, 31, 40, 41]


def brute_force(send, counts, row_elems, recv_cap, sd=None, rd=None):
    """Row placement written out in Python lists, one row at a time."""
    P = len(send)
    out = [[None] * recv_cap for _ in range(P)]
    for s in range(P):
        at = 0
        for d in range(P):
            start = sd[s][d] if sd is not None else at
            at += counts[s][d]
            for i in range(counts[s][d]):
                row = send[s][(start + i) * row_elems:(start + i + 1) * row_elems].tolist()
                if rd is not None:
                    slot = rd[d][s] + i
                else:
                    slot = sum(counts[q][d] for q in range(s)) + i
                assert out[d][slot] is None
                out[d][slot] = row
    return out


@pytest.mark.parametrize("P,row_elems,seed", [(1, 3, 0), (2, 1, 1), (3, 4, 2), (5, 2, 3), (8, 1, 4)])
def test_packed_layout_is_the_brute_force_row_placement(P, row_elems, seed):
    rng = np.random.default_rng(seed)
    counts = rng.integers(0, 4, size=(P, P))
    counts[rng.integers(0, P), rng.integers(0, P)] = 0
    send_cap = int(counts.sum(axis=1).max()) + 2
    recv_cap = int(counts.sum(axis=0).max()) + 1
    send = [rng.integers(-1000, 1000, size=send_cap * row_elems).astype(np.int32) for _ in range(P)]
    recv = [np.full(recv_cap * row_elems, SENTINEL, np.int32) for _ in range(P)]
    ok, rcounts = oracle.alltoallv_dynamic(send, counts, recv, row_elems, send_cap, recv_cap)
    assert ok
    assert np.array_equal(rcounts, counts.T)
    want = brute_force(send, counts.tolist(), row_elems, recv_cap)
    for d in range(P):
        got = rows_of(recv[d], row_elems)
        for slot in range(recv_cap):
            expect = want[d][slot] if want[d][slot] is not None else [SENTINEL] * row_elems
            assert got[slot].tolist() == expect, (d, slot)


@pytest.mark.parametrize("seed", range(4))
def test_explicit_layout_matches_the_static_alltoallv_in_elements(seed):
    rng = np.random.default_rng(100 + seed)
    P, R = 4, 3
    counts = rng.integers(0, 5, size=(P, P))
    # send ranges anywhere (they may overlap: they are only read)
    send_cap = 12
    sd = np.array([[rng.integers(0, send_cap - counts[s, d] + 1) for d in range(P)] for s in range(P)])
    # receive ranges with gaps, shuffled source order
    rd = np.zeros((P, P), np.int64)
    recv_cap = 0
    for d in range(P):
        at = 1
        for s in rng.permutation(P):
            rd[d, s] = at
            at += counts[s, d] + int(rng.integers(0, 2))
        recv_cap = max(recv_cap, at)
    send = [rng.integers(0, 1 << 15, size=send_cap * R).astype(np.uint16) for _ in range(P)]
    recv = [np.full(recv_cap * R, 0xFFFF, np.uint16) for _ in range(P)]
    ok, _ = oracle.alltoallv_dynamic(send, counts, recv, R, send_cap, recv_cap, sdispls=sd, rdispls=rd)
    assert ok
    ref = [np.full(recv_cap * R, 0xFFFF, np.uint16) for _ in range(P)]
    oracle.alltoallv(send, counts * R, sd * R, ref, counts.T * R, rd * R)
    for d in range(P):
        assert np.array_equal(recv[d], ref[d])
    want = brute_force(send, counts.tolist(), R, recv_cap, sd.tolist(), rd.tolist())
    for d in range(P):
        got = rows_of(recv[d], R)
        for slot in range(recv_cap):
            if want[d][slot] is not None:
                assert got[slot].tolist() == want[d][slot]


def _layout_ok(counts, send_cap, recv_cap, sd=None, rd=None, R=1):
    P = len(counts)
    send = [np.arange(send_cap * R, dtype=np.int32) + 100 * s for s in range(P)]
    recv = [np.full(recv_cap * R, SENTINEL, np.int32) for _ in range(P)]
    ok, rc = oracle.alltoallv_dynamic(send, np.array(counts), recv, R, send_cap, recv_cap, sdispls=sd, rdispls=rd)
    if not ok:
        assert all((r == SENTINEL).all() for r in recv), "a rejected layout wrote receive data"
    assert np.array_equal(rc, np.array(counts).T), "recvcounts must be written even when rejected"
    return ok


def test_capacity_boundaries_packed():
    counts = [[2, 3], [1, 1]]
    assert _layout_ok(counts, send_cap=5, recv_cap=4)       # exact fit on both sides
    assert not _layout_ok(counts, send_cap=4, recv_cap=4)   # source 0 needs 5 rows
    assert not _layout_ok(counts, send_cap=5, recv_cap=3)   # rank 1 receives 4 rows


def test_capacity_boundaries_explicit():
    counts = [[2, 0], [0, 3]]
    assert _layout_ok(counts, 5, 5, sd=[[3, 0], [0, 2]], rd=[[3, 0], [0, 2]])
    assert not _layout_ok(counts, 5, 5, sd=[[4, 0], [0, 2]], rd=[[3, 0], [0, 2]])
    assert not _layout_ok(counts, 5, 5, sd=[[3, 0], [0, 2]], rd=[[3, 0], [0, 3]])
    assert not _layout_ok(counts, 5, 5, sd=[[-1, 0], [0, 2]], rd=[[3, 0], [0, 2]])


def test_negative_count_is_rejected():
    assert not _layout_ok([[1, -1], [0, 0]], 8, 8)


def test_receive_overlap_boundaries():
    counts = [[2, 0], [2, 0]]
    assert _layout_ok(counts, 4, 4, sd=[[0, 0], [0, 0]], rd=[[0, 2], [0, 0]])        # adjacent
    assert not _layout_ok(counts, 4, 4, sd=[[0, 0], [0, 0]], rd=[[0, 1], [0, 0]])    # one row shared
    assert not _layout_ok(counts, 4, 4, sd=[[0, 0], [0, 0]], rd=[[1, 0], [0, 0]])    # other side


def test_zero_count_ranges_are_never_checked():
    counts = [[0, 1], [0, 0]]
    assert _layout_ok(counts, 1, 1, sd=[[1 << 40, 0], [-5, 7]], rd=[[-3, 99], [0, 1 << 50]])


def test_send_ranges_may_overlap():
    counts = [[2, 2], [0, 0]]
    assert _layout_ok(counts, 2, 2, sd=[[0, 0], [0, 0]], rd=[[0, 0], [0, 0]])


def test_empty_exchange():
    P = 3
    counts = np.zeros((P, P), np.int64)
    assert _layout_ok(counts.tolist(), 0, 0)
