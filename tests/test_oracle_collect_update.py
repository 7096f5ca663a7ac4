"""Pins for the oracle's collection, priority update and ring insertion.

Collection reads a range of timesteps of a subset of fields from column
tables whose blocks hold one field of one trajectory (GEAR Sec. 3.2 storage
format, Sec. 3.4 collection example).  The update writes status-table
priorities (Sec. 3.2).  Insertion overwrites the oldest trajectory once the
store is full (Sec. 3.2, insertion and deletion).  The checks compare with
numpy fancy indexing and numpy formulations of "last write wins".
"""
import numpy as np
import pytest

import oracle
from gen import STAMP, Column, fill_rows_cpu


@pytest.mark.parametrize("E", [1, 4, 17, 68, 1024])
def test_collect_matches_numpy_fancy_indexing(E):
    rng = np.random.default_rng(E)
    N, T, L, B = 37, 23, 5, 64
    tab = rng.integers(0, 256, size=(N, T, E), dtype=np.uint8)
    idx = rng.integers(0, N, size=B)
    start = rng.integers(0, T - L + 1, size=B).astype(np.int32)
    st, outs = oracle.collect([tab], T, idx, start, L)
    assert st == oracle.OK
    ref = tab[idx[:, None], start[:, None] + np.arange(L)[None, :]].reshape(B, L * E)
    np.testing.assert_array_equal(outs[0], ref)


def test_collect_full_trajectory_is_block_copy():
    rng = np.random.default_rng(2)
    N, T, E = 9, 16, 12
    tab = rng.integers(0, 256, size=(N, T * E), dtype=np.uint8)
    idx = np.array([3, 3, 0, 8, 5])
    st, outs = oracle.collect([tab], T, idx, np.zeros(5, np.int32), T)
    assert st == oracle.OK
    np.testing.assert_array_equal(outs[0], tab[idx])


def test_collect_several_columns_and_stamps():
    N, T, L, B = 50, 40, 9, 33
    col = Column("stamp", STAMP, 1)
    rows = fill_rows_cpu(col, 0, 0, T, 0, N)
    other = np.random.default_rng(4).integers(0, 256, size=(N, T * 3), dtype=np.uint8)
    rng = np.random.default_rng(5)
    idx = rng.integers(0, N, size=B)
    start = rng.integers(0, T - L + 1, size=B).astype(np.int32)
    st, outs = oracle.collect([rows, other], T, idx, start, L)
    assert st == oracle.OK
    kt = outs[0].view(np.uint32).reshape(B, L, 2)
    np.testing.assert_array_equal(kt[:, :, 0], np.repeat(idx[:, None], L, axis=1))
    np.testing.assert_array_equal(kt[:, :, 1], start[:, None] + np.arange(L)[None, :])
    np.testing.assert_array_equal(outs[1], other.reshape(N, T, 3)[idx[:, None], start[:, None] + np.arange(L)].reshape(B, -1))


def test_collect_rejects_out_of_range():
    tab = np.zeros((4, 10), dtype=np.uint8)
    assert oracle.collect([tab], 10, [4], [0], 3)[0] == oracle.INVAL
    assert oracle.collect([tab], 10, [-2], [0], 3)[0] == oracle.INVAL
    assert oracle.collect([tab], 10, [1], [8], 3)[0] == oracle.INVAL
    assert oracle.collect([tab], 10, [1], [7], 3)[0] == oracle.OK


def test_collect_index_minus_one_is_an_empty_window():
    # -1 marks a draw with no trajectory: its window is zeros, whatever start.
    tab = np.arange(40, dtype=np.uint8).reshape(4, 10) + 1
    st, outs = oracle.collect([tab], 10, [2, -1, 0], [1, 99, 7], 3)
    assert st == oracle.OK
    np.testing.assert_array_equal(outs[0], [[22, 23, 24], [0, 0, 0], [8, 9, 10]])


def test_update_last_occurrence_wins():
    rng = np.random.default_rng(6)
    N, B = 100, 5000
    p = rng.integers(1, 1000, size=N).astype(np.uint32)
    old = p.copy()
    idx = rng.integers(0, N, size=B)
    newp = rng.integers(1, 1000, size=B).astype(np.uint32)
    assert oracle.update(p, idx, newp) == oracle.OK
    # numpy formulation: the last position of each slot in the batch.
    rev_slots, rev_first = np.unique(idx[::-1], return_index=True)
    last_pos = B - 1 - rev_first
    expect = old.copy()
    expect[rev_slots] = newp[last_pos]
    np.testing.assert_array_equal(p, expect)
    delta = int(newp[last_pos].astype(np.int64).sum() - old[rev_slots].astype(np.int64).sum())
    assert int(p.astype(np.int64).sum()) - int(old.astype(np.int64).sum()) == delta


def test_update_rejects_out_of_range_and_is_atomic():
    p = np.arange(10, dtype=np.uint32)
    before = p.copy()
    assert oracle.update(p, [1, 10], [5, 5]) == oracle.INVAL
    np.testing.assert_array_equal(p, before)


def test_insert_ring_keeps_last_N():
    N, T = 8, 3
    col = Column("stamp", STAMP, 1)
    store = oracle.Store([col.elem_bytes], N, T)
    total = 0
    for n in [3, 4, 9, 1, 20]:
        rows = fill_rows_cpu(col, 0, 0, T, total, n)
        store.insert([rows], np.arange(total, total + n, dtype=np.uint32) + 1)
        total += n
        assert store.next_seq == total
        live = min(total, N)
        ks = store.cols[0].view(np.uint32).reshape(N, T, 2)[:, 0, 0]
        for k in range(total - live, total):
            assert ks[k % N] == k
            assert store.priority[k % N] == k + 1
