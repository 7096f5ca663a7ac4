"""Pins for the oracle's index manager (GEAR Sec. 3.2: a block allocator with
one free-index queue, a status table whose priority is 0 for indices that are
free or being written, allocate / commit insertion, and FIFO or LIFO removal
of a victim when no index is free or the selectable count reaches the preset
maximum).

The checks compare it with the oracle's independent ring insertion (FIFO
removal at capacity N is the ring), with commit and release times recorded
by the tests themselves, with invariants over random operation sequences,
and with a worked example.
"""
import numpy as np
import pytest

import oracle
from gen import STAMP, Column, fill_rows_cpu


def _stamp_rows(k0, n, T=4):
    return [fill_rows_cpu(Column("stamp", STAMP, 1), 0, 0, T, k0, n)]


@pytest.mark.parametrize("chunk", [1, 3, 16])
def test_fifo_allocator_at_capacity_is_the_ring(chunk):
    # Same rows and priorities through the ring and through allocate/commit.
    N, T, total = 16, 4, 61
    ring = oracle.Store([8], N, T)
    im = oracle.Store([8], N, T)
    im.use_allocator(oracle.FIFO, N)
    rng = np.random.default_rng(chunk)
    k = 0
    while k < total:
        n = min(chunk, total - k)
        prio = rng.integers(1, 1000, size=n).astype(np.uint32)
        rows = _stamp_rows(k, n, T)
        ring.insert(rows, prio)
        assert im.insert(rows, prio) == oracle.OK
        k += n
        np.testing.assert_array_equal(im.priority, ring.priority)
        np.testing.assert_array_equal(im.cols[0], ring.cols[0])
        live = min(k, N)
        # The committed list is the ring's live slots, oldest insertion first.
        np.testing.assert_array_equal(im.im.order(), (np.arange(k - live, k) % N))
        for strat in (oracle.FIFO, oracle.LIFO, oracle.PRIORITIZED, oracle.TOPK):
            B = min(live, 5)
            a = ring.select(strat, B, 2, 99 + k, 0.4, True)
            b = im.select(strat, B, 2, 99 + k, 0.4, True)
            assert a[0] == b[0]
            for x, y in zip(a[1:], b[1:]):
                np.testing.assert_array_equal(x, y)
        # Uniform: the same draw r picks live slot r of the ring and the
        # r-th oldest committed index of the manager.
        a = ring.select(oracle.UNIFORM, 40, 2, 7 + k)
        b = im.select(oracle.UNIFORM, 40, 2, 7 + k)
        order = im.im.order()
        oldest = (k - live) % N
        np.testing.assert_array_equal(b[1], order[(a[1] - 0)])  # r-th committed
        np.testing.assert_array_equal(b[1], (oldest + a[1]) % N if k > N else a[1])


def test_lifo_releases_the_newest_commit():
    N, M = 8, 5
    m = oracle.IndexManager(N, oracle.LIFO, M)
    p = np.zeros(N, dtype=np.uint32)
    st, a = m.allocate(5, p)
    assert st == oracle.OK and list(a) == [0, 1, 2, 3, 4]
    assert m.commit([3, 0, 4, 1, 2], [10, 11, 12, 13, 14], p) == oracle.OK   # commit order 3,0,4,1,2
    st, b = m.allocate(1, p)       # 5 selectable = maximum: release the newest commit (2)
    assert st == oracle.OK
    assert p[2] == 0 and list(m.order()) == [3, 0, 4, 1]
    # Free queue was [5,6,7] then 2 joined its back: the front (5) is allocated.
    assert list(b) == [5] and list(m.free_queue()) == [6, 7, 2]
    assert m.commit(b, [20], p) == oracle.OK
    st, c = m.allocate(2, p)       # releases 5 (newest) then 1
    assert st == oracle.OK and list(c) == [6, 7]
    assert list(m.order()) == [3, 0, 4] and p[5] == 0 and p[1] == 0
    assert list(m.free_queue()) == [2, 5, 1]


def test_fifo_releases_the_oldest_commit_and_reuses_released_first():
    N, M = 6, 4
    m = oracle.IndexManager(N, oracle.FIFO, M)
    p = np.zeros(N, dtype=np.uint32)
    _, a = m.allocate(4, p)
    m.commit([2, 1, 3, 0], [5, 6, 7, 8], p)     # oldest commit: 2
    _, b = m.allocate(2, p)        # releases 2 then 1; free queue [4,5,2,1]: hands out 4, 5
    assert list(b) == [4, 5] and list(m.free_queue()) == [2, 1]
    assert p[2] == 0 and p[1] == 0 and list(m.order()) == [3, 0]
    m.commit([5, 4], [9, 9], p)
    _, c = m.allocate(3, p)        # 4 selectable: releases 3, 0, 5; hands out 2, 1, 3
    assert list(c) == [2, 1, 3] and list(m.order()) == [4]


def test_pending_indices_are_never_released():
    N = 4
    m = oracle.IndexManager(N, oracle.FIFO, 3)
    p = np.zeros(N, dtype=np.uint32)
    st, a = m.allocate(3, p)
    assert st == oracle.OK
    st, b = m.allocate(1, p)       # 3 pending = maximum: nothing can be released
    assert st == oracle.INSUFFICIENT and b.size == 1 and m.n_pending == 3
    assert m.commit(a[:1], [1], p) == oracle.OK
    st, b = m.allocate(1, p)       # still 2 pending + 1 committed: release the committed one
    assert st == oracle.OK and p[a[0]] == 0


def test_commit_rejects_bad_lists_without_change():
    m = oracle.IndexManager(8, oracle.FIFO, 8)
    p = np.zeros(8, dtype=np.uint32)
    _, a = m.allocate(3, p)
    assert m.commit([a[0], a[0]], [1, 1], p) == oracle.INVAL     # duplicate
    assert m.commit([a[0], 7], [1, 1], p) == oracle.INVAL        # 7 is free, not pending
    assert m.commit([a[0], -1], [1, 1], p) == oracle.INVAL
    assert m.n_pending == 3 and m.n_committed == 0 and not p.any()


def test_update_skips_indices_that_are_not_committed():
    m = oracle.IndexManager(6, oracle.FIFO, 6)
    p = np.zeros(6, dtype=np.uint32)
    _, a = m.allocate(4, p)
    m.commit(a[:2], [5, 6], p)
    assert m.update(p, [a[0], a[2], 5, a[1], a[0]], [50, 60, 70, 80, 90]) == oracle.OK
    assert p[a[0]] == 90 and p[a[1]] == 80 and p[a[2]] == 0 and p[5] == 0
    assert m.update(p, [6], [1]) == oracle.INVAL


@pytest.mark.parametrize("removal,seed", [(oracle.FIFO, 1), (oracle.LIFO, 2), (oracle.FIFO, 3), (oracle.LIFO, 4)])
def test_random_sequences_keep_the_invariants(removal, seed):
    rng = np.random.default_rng(seed)
    N = 40
    M = int(rng.integers(5, N + 1))
    m = oracle.IndexManager(N, removal, M)
    p = np.zeros(N, dtype=np.uint32)
    pending = []
    commit_time = {}
    release_time = {}
    clock = 0
    for step in range(400):
        op = rng.integers(0, 3)
        if op == 0:
            n = int(rng.integers(1, 6))
            before = set(m.order().tolist())
            st, idx = m.allocate(n, p)
            if len(pending) + n > M:
                assert st == oracle.INSUFFICIENT
                continue
            assert st == oracle.OK
            after = set(m.order().tolist())
            released = before - after
            # Victims: exactly the oldest (FIFO) / newest (LIFO) commits.
            need = max(0, len(before) + len(pending) + n - M)
            assert len(released) == need
            ranked = sorted(before, key=lambda i: commit_time[i], reverse=(removal == oracle.LIFO))
            assert released == set(ranked[:need])
            for v in ranked[:need]:         # released in that order
                clock += 1
                release_time[v] = clock
                del commit_time[v]
            # Allocation hands out never-used indices in index order, then
            # released ones in release order.
            fresh = [i for i in idx if i not in release_time]
            assert fresh == sorted(fresh)
            reused = [i for i in idx if i in release_time]
            assert reused == sorted(reused, key=lambda i: release_time[i])
            for i in idx:
                release_time.pop(i, None)
            pending += idx.tolist()
        elif op == 1 and pending:
            k = int(rng.integers(1, len(pending) + 1))
            pick = [pending[j] for j in rng.permutation(len(pending))[:k]]
            prio = rng.integers(1, 100, size=k).astype(np.uint32)
            assert m.commit(pick, prio, p) == oracle.OK
            for i in pick:
                clock += 1
                commit_time[i] = clock
                pending.remove(i)
            np.testing.assert_array_equal(p[pick], prio)
        elif op == 2:
            idx = rng.integers(0, N, size=6)
            assert m.update(p, idx, rng.integers(1, 100, size=6).astype(np.uint32)) == oracle.OK
        order = m.order()
        assert list(order) == sorted(commit_time, key=lambda i: commit_time[i])
        assert m.n_committed + m.n_pending <= M and m.n_pending == len(pending)
        assert m.n_committed + m.n_pending + m.n_free == N
        st_ = m.state()
        assert set(np.nonzero(st_ == oracle.IM_COMMITTED)[0]) == set(commit_time)
        assert set(np.nonzero(st_ == oracle.IM_PENDING)[0]) == set(pending)
        nz = set(np.nonzero(p)[0].tolist())
        assert nz <= set(commit_time)          # only committed indices are selectable


def test_select_on_the_committed_list():
    # FIFO/LIFO/uniform pick from the committed list; prioritized and TopK see
    # zero priority on everything else.
    N = 10
    s = oracle.Store([], N, 4)
    s.use_allocator(oracle.LIFO, 6)
    st, a = s.allocate(6)
    s.commit([a[4], a[1], a[5]], [3, 9, 1])
    st, idx, _, _ = s.select(oracle.FIFO, 3, 2, 0)
    assert st == oracle.OK and list(idx) == [a[4], a[1], a[5]]
    st, idx, _, _ = s.select(oracle.LIFO, 2, 2, 0)
    assert list(idx) == [a[5], a[1]]
    assert s.select(oracle.FIFO, 4, 2, 0)[0] == oracle.INSUFFICIENT
    st, idx, _, _ = s.select(oracle.UNIFORM, 500, 2, 5)
    assert set(idx.tolist()) == {a[4], a[1], a[5]}
    st, idx, _, _ = s.select(oracle.TOPK, 4, 2, 0)
    assert st == oracle.NO_WEIGHT and list(idx) == [a[1], a[4], a[5], -1]
    st, idx, _, _ = s.select(oracle.PRIORITIZED, 200, 2, 3)
    assert set(idx.tolist()) == {a[4], a[1], a[5]}
    empty = oracle.Store([], N, 4)
    empty.use_allocator(oracle.FIFO, N)
    empty.allocate(3)
    assert empty.select(oracle.UNIFORM, 1, 1, 0)[0] == oracle.EMPTY
