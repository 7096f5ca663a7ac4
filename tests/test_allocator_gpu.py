"""GPU parity of the index manager (GEAR Sec. 3.2: allocate -> in-place
writes -> commit, a free-index queue, FIFO or LIFO removal at a preset
maximum; priority zero for indices that are free or being written).

Every step is compared with the oracle's index manager: the allocated
indices, the priorities (bit-exact), the counts, and every few steps all
five strategies and the collected windows.
"""
import numpy as np
import pytest
import torch

import gen
import oracle
from paper_2310_05205_amd import gear
from tests.helpers import DEV, cuda, host, say

pytestmark = pytest.mark.gpu

COLS = (gen.Column("stamp", gen.STAMP, 1), gen.Column("obs", gen.NORMAL_F32, 5))


def _rows(ks, T, seed=7):
    return [gen.fill_rows_list_cpu(c, ci, seed, T, np.asarray(ks, dtype=np.int64)) for ci, c in enumerate(COLS)]


def _write(t, idx, rows):
    """In-place writes of the rows into the allocated blocks, through the
    column views (device tensor or pinned host array)."""
    for c, r in enumerate(rows):
        view = t.column_view(c)
        r = np.ascontiguousarray(r).reshape(len(idx), -1).view(np.uint8)
        if isinstance(view, np.ndarray):
            torch.cuda.synchronize(DEV)       # earlier stream work on these blocks is done
            view[np.asarray(idx)] = r
        else:
            view[torch.from_numpy(np.asarray(idx)).to(cuda())] = torch.from_numpy(r).to(cuda())


def _check_state(t, store, where):
    torch.cuda.synchronize(DEV)
    np.testing.assert_array_equal(t.priorities(), store.priority, err_msg=where)
    im = store.im
    assert t.allocator_info() == (im.n_committed, im.n_pending, im.n_free), where
    assert t.info()[0] == im.n_committed


def _check_selects(t, store, it, T):
    live = store.im.n_committed
    if live == 0:
        with pytest.raises(gear.GearError) as e:
            t.select(gear.GEAR_UNIFORM, 4, 1, it)
        assert e.value.code == gear.GEAR_E_EMPTY
        return
    L = 1 + it % T
    for strat in (gear.GEAR_FIFO, gear.GEAR_LIFO, gear.GEAR_UNIFORM, gear.GEAR_PRIORITIZED, gear.GEAR_TOPK):
        B = min(live, 7) if strat in (gear.GEAR_FIFO, gear.GEAR_LIFO) else 64
        seed = gen.select_seed(11, it * 8 + strat)
        st, oidx, ostart, ow = store.select(strat, B, L, seed, 0.5, True)
        if st == oracle.NO_WEIGHT and strat == gear.GEAR_PRIORITIZED:
            continue
        idx, start, w = t.select(strat, B, L, seed, 0.5, weights=True)
        np.testing.assert_array_equal(host(idx), oidx, err_msg="strategy %d" % strat)
        np.testing.assert_array_equal(host(start), ostart)
        np.testing.assert_allclose(host(w).astype(np.float64), ow.astype(np.float64), rtol=1e-6, atol=0)
        sel = oidx >= 0
        if sel.any():
            outs = t.collect(idx[torch.from_numpy(sel).to(cuda())], start[torch.from_numpy(sel).to(cuda())], L)
            st2, oouts = store.collect(oidx[sel], ostart[sel], L)
            assert st2 == oracle.OK
            for a, b in zip(outs, oouts):
                np.testing.assert_array_equal(host(a), b)
    assert t.sync() in (0, gear.GEAR_STATUS_NO_WEIGHT)


SEQ_CASES = [(gear.GEAR_FIFO, 200, 200, 1), (gear.GEAR_LIFO, 200, 120, 2), (gear.GEAR_FIFO, 300, 50, 3),
             (gear.GEAR_LIFO, 64, 64, 4)]


@pytest.mark.parametrize("removal,N,M,seed", SEQ_CASES, ids=["fifo-full", "lifo-max120", "fifo-max50", "lifo-64"])
@pytest.mark.parametrize("residency", [gear.GEAR_DEVICE, gear.GEAR_HOST_PINNED], ids=["hbm", "pinned"])
def test_random_operation_sequences(removal, N, M, seed, residency):
    T = 6
    rng = np.random.default_rng(seed)
    eb = [c.elem_bytes for c in COLS]
    t = gear.Table(eb, N, T, residency, DEV)
    store = oracle.Store(eb, N, T)
    try:
        t.use_allocator(removal, M)
        store.use_allocator(removal, M)
        pending = []
        k = 0
        for it in range(120):
            say("allocator seq removal=%d N=%d M=%d step %d" % (removal, N, M, it))
            op = rng.integers(0, 4)
            if op <= 1:
                n = int(rng.integers(1, max(2, M // 3)))
                st, oidx = store.allocate(n)
                if st == oracle.INSUFFICIENT:
                    with pytest.raises(gear.GearError) as e:
                        t.allocate(n)
                    assert e.value.code == gear.GEAR_E_INSUFFICIENT
                    continue
                idx = t.allocate(n)
                np.testing.assert_array_equal(idx, oidx)
                rows = _rows(np.arange(k, k + n), T)
                k += n
                _write(t, idx, rows)
                store.write(idx, rows)
                pending += idx.tolist()
            elif op == 2 and pending:
                m = int(rng.integers(1, len(pending) + 1))
                pick = np.array([pending[j] for j in rng.permutation(len(pending))[:m]], dtype=np.int64)
                prio = rng.integers(0, 50, size=m).astype(np.uint32)    # 0 commits an unselectable index
                # priorities from device memory and pinned host memory (read in
                # place by the commit kernel) or pageable memory (staged)
                src = int(rng.integers(0, 3))
                if src == 0:
                    t.commit(pick, torch.from_numpy(prio).to(cuda()))
                elif src == 1:
                    t.commit(pick, torch.from_numpy(prio.view(np.int32)).pin_memory())
                else:
                    t.commit(pick, prio)
                assert store.commit(pick, prio) == oracle.OK
                for i in pick:
                    pending.remove(int(i))
            else:
                B = int(rng.integers(1, 40))
                uidx = rng.integers(0, N, size=B).astype(np.int64)
                newp = rng.integers(1, 1000, size=B).astype(np.uint32)
                t.update_priorities(torch.from_numpy(uidx).to(cuda()), torch.from_numpy(newp).to(cuda()))
                assert store.update(uidx, newp) == oracle.OK
            _check_state(t, store, "step %d" % it)
            if it % 10 == 9:
                _check_selects(t, store, it, T)
    finally:
        t.close()


@pytest.mark.parametrize("residency", [gear.GEAR_DEVICE, gear.GEAR_HOST_PINNED], ids=["hbm", "pinned"])
@pytest.mark.parametrize("removal", [gear.GEAR_FIFO, gear.GEAR_LIFO], ids=["fifo", "lifo"])
def test_managed_insert_matches_oracle(residency, removal):
    N, T, M = 1000, 4, 700
    eb = [c.elem_bytes for c in COLS]
    t = gear.Table(eb, N, T, residency, DEV)
    store = oracle.Store(eb, N, T)
    try:
        t.use_allocator(removal, M)
        store.use_allocator(removal, M)
        k = 0
        for it, n in enumerate([300, 250, 400, 1, 699, 3]):
            say("managed insert removal=%d batch %d" % (removal, it))
            rows = _rows(np.arange(k, k + n), T)
            prio = gen.insert_priorities(gen.PrioDist(gen.PRIO_UNIFORM, 1, 1000), 5, k, n)
            k += n
            t.insert([np.ascontiguousarray(r) for r in rows], prio)
            assert store.insert(rows, prio) == oracle.OK
            _check_state(t, store, "insert %d" % it)
            _check_selects(t, store, it, T)
        with pytest.raises(gear.GearError) as e:       # more than the maximum at once
            t.insert([np.ascontiguousarray(r) for r in _rows(np.arange(M + 1), T)], np.ones(M + 1, np.uint32))
        assert e.value.code == gear.GEAR_E_INSUFFICIENT
    finally:
        t.close()


def test_lists_longer_than_one_staging_chunk():
    # 200k indices per call (several 65536-entry chunks), churn through LIFO
    # removal, then the prioritized select and TopK over the result.
    N, T, M = 1 << 18, 1, 150000
    t = gear.Table([], N, T, gear.GEAR_DEVICE, DEV)
    store = oracle.Store([], N, T)
    try:
        t.set_options(gear.GEAR_OPT_INCREMENTAL_TREE)
        t.use_allocator(gear.GEAR_LIFO, M)
        store.use_allocator(gear.GEAR_LIFO, M)
        rng = np.random.default_rng(9)
        for it, (n, m) in enumerate([(140000, 140000), (100000, 60000), (150000 - 40000, 110000 - 60000)]):
            say("staging chunks step %d" % it)
            st, oidx = store.allocate(n)
            assert st == oracle.OK
            idx = t.allocate(n)
            np.testing.assert_array_equal(idx, oidx)
            pend = store.im.state() == oracle.IM_PENDING
            pick = np.nonzero(pend)[0][rng.permutation(int(pend.sum()))[:m]].astype(np.int64)
            prio = rng.integers(1, 1 << 20, size=pick.size).astype(np.uint32)
            t.commit(pick, prio)
            assert store.commit(pick, prio) == oracle.OK
            _check_state(t, store, "chunk step %d" % it)
            B = 8192
            uidx = rng.integers(0, N, size=B).astype(np.int64)
            newp = rng.integers(1, 1 << 20, size=B).astype(np.uint32)
            t.update_priorities(torch.from_numpy(uidx).to(cuda()), torch.from_numpy(newp).to(cuda()))
            store.update(uidx, newp)
            for strat in (gear.GEAR_PRIORITIZED, gear.GEAR_TOPK, gear.GEAR_UNIFORM, gear.GEAR_LIFO):
                seed = gen.select_seed(3, it * 4 + strat)
                st, oi, os_, ow = store.select(strat, 4096, 1, seed, 0.4, True)
                i_, s_, w_ = t.select(strat, 4096, 1, seed, 0.4, weights=True)
                np.testing.assert_array_equal(host(i_), oi)
                np.testing.assert_allclose(host(w_).astype(np.float64), ow.astype(np.float64), rtol=1e-6, atol=0)
            assert t.sync() == 0
    finally:
        t.close()


def test_allocator_errors():
    t = gear.Table([4], 16, 2, gear.GEAR_DEVICE, DEV)
    try:
        with pytest.raises(gear.GearError):
            t.allocate(1)                              # no index manager yet
        with pytest.raises(gear.GearError):
            t.use_allocator(7, 8)                      # removal must be FIFO or LIFO
        with pytest.raises(gear.GearError):
            t.use_allocator(gear.GEAR_FIFO, 17)        # above capacity
        t.use_allocator(gear.GEAR_FIFO, 8)
        with pytest.raises(gear.GearError):
            t.use_allocator(gear.GEAR_FIFO, 8)         # already managed
        idx = t.allocate(3)
        assert list(idx) == [0, 1, 2]
        for bad in ([0, 0], [0, 5], [0, -1]):
            with pytest.raises(gear.GearError) as e:
                t.commit(np.array(bad, np.int64), np.ones(2, np.uint32))
            assert e.value.code == gear.GEAR_E_INVAL
        assert t.allocator_info() == (0, 3, 13)        # nothing changed
        t.commit(idx[::-1].copy(), np.array([3, 2, 1], np.uint32))
        assert t.allocator_info() == (3, 0, 13)
        with pytest.raises(gear.GearError) as e:
            t.allocate(9)
        assert e.value.code == gear.GEAR_E_INSUFFICIENT
        torch.cuda.synchronize(DEV)
        assert list(t.priorities()[:4]) == [1, 2, 3, 0]
    finally:
        t.close()
    r = gear.Table([4], 16, 2, gear.GEAR_DEVICE, DEV)
    try:
        r.insert([np.zeros((1, 8), np.uint8)], np.ones(1, np.uint32))
        with pytest.raises(gear.GearError):
            r.use_allocator(gear.GEAR_FIFO, 8)         # the ring already holds insertions
    finally:
        r.close()


ODD_COLS = (gen.Column("b3", gen.BYTES, 3), gen.Column("w12", gen.INT_MOD, 3, param=7),
            gen.Column("v64", gen.NORMAL_F32, 16))


@pytest.mark.parametrize("source", ["device", "pinned", "device-misaligned"])
@pytest.mark.parametrize("residency", [gear.GEAR_DEVICE, gear.GEAR_HOST_PINNED], ids=["hbm", "pinned"])
def test_row_scatter_kernel_paths(source, residency):
    # gear_insert with LIFO removal (victims released newest first, so slots
    # come in descending order) from device-readable sources: the scatter
    # kernel with 16-, 4- and 1-byte elements (rows of 48, 36... bytes, and a
    # source one byte off alignment).
    N, T, M = 700, 3, 500
    eb = [c.elem_bytes for c in ODD_COLS]
    t = gear.Table(eb, N, T, residency, DEV)
    store = oracle.Store(eb, N, T)
    try:
        t.use_allocator(gear.GEAR_LIFO, M)
        store.use_allocator(oracle.LIFO, M)
        k = 0
        for it, n in enumerate([500, 300, 499, 7]):
            say("row scatter %s residency=%d batch %d" % (source, residency, it))
            rows = [gen.fill_rows_list_cpu(c, ci, 9, T, np.arange(k, k + n)) for ci, c in enumerate(ODD_COLS)]
            prio = gen.insert_priorities(U1000, 9, k, n)
            k += n
            if source == "pinned":
                srcs = [torch.from_numpy(r).pin_memory() for r in rows]
            elif source == "device":
                srcs = [torch.from_numpy(r).to(cuda()) for r in rows]
            else:
                bufs = [torch.zeros(r.size + 1, dtype=torch.uint8, device=cuda()) for r in rows]
                for b_, r in zip(bufs, rows):
                    b_[1:] = torch.from_numpy(r.reshape(-1)).to(cuda())
                srcs = [b_[1:] for b_ in bufs]
            t.insert(srcs, prio)
            assert store.insert(rows, prio) == oracle.OK
            torch.cuda.synchronize(DEV)
            for c in range(len(ODD_COLS)):
                view = t.column_view(c)
                got = view if isinstance(view, np.ndarray) else host(view)
                np.testing.assert_array_equal(got, store.cols[c], err_msg="column %d" % c)
            _check_state(t, store, "batch %d" % it)
    finally:
        t.close()


U1000 = gen.PrioDist(gen.PRIO_UNIFORM, 1, 1000)


def test_write_rows_on_a_ring_table():
    # Writes into arbitrary slots of a ring table, any order, then collect.
    N, T = 300, 4
    eb = [c.elem_bytes for c in COLS]
    t = gear.Table(eb, N, T, gear.GEAR_DEVICE, DEV)
    store = oracle.Store(eb, N, T)
    try:
        prio = np.arange(1, N + 1, dtype=np.uint32)
        rows0 = _rows(np.arange(N), T)
        t.insert([np.ascontiguousarray(r) for r in rows0], prio)
        store.insert(rows0, prio)
        rng = np.random.default_rng(5)
        slots = rng.permutation(N)[:120].astype(np.int64)
        rows = _rows(np.arange(1000, 1120), T)
        t.write_rows(slots, [torch.from_numpy(np.ascontiguousarray(r)).to(cuda()) for r in rows])
        store.write(slots, rows)
        idx = torch.from_numpy(rng.integers(0, N, size=256).astype(np.int64)).to(cuda())
        start = torch.zeros(256, dtype=torch.int32, device=cuda())
        outs = t.collect(idx, start, T)
        st, oouts = store.collect(host(idx), host(start), T)
        for a, b in zip(outs, oouts):
            np.testing.assert_array_equal(host(a), b)
        with pytest.raises(gear.GearError):
            t.write_rows(np.array([N], np.int64), [torch.zeros(T * e, dtype=torch.uint8, device=cuda()) for e in eb])
        assert t.sync() == 0
    finally:
        t.close()


def test_new_tables_read_zero_after_reuse():
    # Freed pinned (and device) memory can come back with old contents; a new
    # table must still read as zeros in every slot never written.
    for residency in (gear.GEAR_HOST_PINNED, gear.GEAR_DEVICE):
        for _ in range(3):
            t = gear.Table([40], 2000, 5, residency, DEV)
            v = t.column_view(0)
            if isinstance(v, np.ndarray):
                assert not v.any()
                v[:] = 0xFF
            else:
                assert int(v.count_nonzero()) == 0
                v.fill_(0xFF)
            torch.cuda.synchronize(DEV)
            t.close()
