"""Allocation failures leave no table behind and leak nothing.

GEAR_TEST_FAIL_ALLOC=n makes the n-th allocation of one gear_table_create
or gear_table_use_allocator call fail as if memory were exhausted (a plain
allocation failure: nothing reaches a kernel).  Every allocation of both
calls is made to fail in turn; each must return GEAR_E_NOMEM, free what the
call had allocated, and leave the device able to create and use tables.  A
table larger than HBM fails the same way without the hook."""
import os

import numpy as np
import pytest
import torch

from paper_2310_05205_amd import gear
from tests.helpers import cuda, host, say

pytestmark = pytest.mark.gpu


@pytest.fixture
def fail_at():
    def set_n(n):
        if n is None:
            os.environ.pop("GEAR_TEST_FAIL_ALLOC", None)
        else:
            os.environ["GEAR_TEST_FAIL_ALLOC"] = str(n)
    yield set_n
    os.environ.pop("GEAR_TEST_FAIL_ALLOC", None)


def _free_bytes():
    torch.cuda.synchronize()
    return torch.cuda.mem_get_info(0)[0]


def _usable(residency):
    """A small table works end to end: insert, select, collect, update."""
    t = gear.Table([8, 4], 64, 4, residency, 0)
    try:
        rows = [np.arange(64 * 4 * 8, dtype=np.uint8).reshape(64, 32), np.ones((64, 16), np.uint8)]
        t.insert(rows, np.arange(1, 65, dtype=np.uint32))
        idx, start, w = t.select(gear.GEAR_PRIORITIZED, 16, 2, 7, 0.4, weights=True)
        outs = t.collect(idx, start, 2)
        i, s = host(idx), host(start)
        for b in range(16):
            assert np.array_equal(host(outs[0])[b], rows[0][i[b], s[b] * 8:(s[b] + 2) * 8])
        t.update_priorities(idx, torch.ones(16, dtype=torch.int32, device=cuda()))
        assert t.sync() == 0
    finally:
        t.close()


@pytest.mark.parametrize("residency", [gear.GEAR_DEVICE, gear.GEAR_HOST_PINNED], ids=["device", "pinned"])
def test_every_allocation_of_create_can_fail_cleanly(fail_at, residency):
    # Large enough that a leaked column or priority array would show.
    cols, N, T = [64, 16], 1 << 20, 4
    # One table first, so that memory the runtime sets aside once per
    # process (code objects, pools) is not counted as a leak.
    gear.Table(cols, N, T, residency, 0).close()
    free0 = _free_bytes()
    n = 1
    while True:
        say("create with allocation %d failing (residency %d)" % (n, residency))
        fail_at(n)
        try:
            t = gear.Table(cols, N, T, residency, 0)
        except gear.GearError as e:
            assert e.code == gear.GEAR_E_NOMEM, str(e)
            assert "allocation" in str(e)
            n += 1
            continue
        t.close()   # n is past the call's last allocation: the table was made
        break
    fail_at(None)
    assert n >= 16, n        # columns, priorities, tags, tree, minima, status, staging, TopK scratch
    assert free0 - _free_bytes() < (64 << 20)
    _usable(residency)


def test_every_allocation_of_the_index_manager_can_fail_cleanly(fail_at):
    for n in (1, 2):
        t = gear.Table([4], 1000, 2)
        try:
            fail_at(n)
            with pytest.raises(gear.GearError) as e:
                t.use_allocator(gear.GEAR_FIFO)
            assert e.value.code == gear.GEAR_E_NOMEM
            fail_at(None)
            # Still a ring table, and the index manager can be added afterwards.
            t.use_allocator(gear.GEAR_FIFO)
            idx = t.allocate(10)
            t.commit(idx, np.arange(1, 11, dtype=np.uint32))
            assert t.allocator_info() == (10, 0, 990)
            sel, _, _ = t.select(gear.GEAR_FIFO, 10, 1, 0)
            assert list(host(sel)) == list(idx)
            assert t.sync() == 0
        finally:
            fail_at(None)
            t.close()


def test_an_error_pending_from_another_call_is_not_reported_as_ours():
    # A failed allocation outside the library leaves a HIP error pending in
    # this thread; the next library calls must still succeed.
    with pytest.raises(torch.OutOfMemoryError):
        torch.empty(400 << 30, dtype=torch.uint8, device=cuda())
    _usable(gear.GEAR_DEVICE)


def test_a_table_larger_than_hbm_is_refused():
    _usable(gear.GEAR_DEVICE)
    free0 = _free_bytes()
    with pytest.raises(gear.GearError) as e:
        gear.Table([400], 1 << 30, 1, gear.GEAR_DEVICE, 0)     # 400 GB of columns
    assert e.value.code == gear.GEAR_E_NOMEM
    assert free0 - _free_bytes() < (64 << 20)
    _usable(gear.GEAR_DEVICE)
