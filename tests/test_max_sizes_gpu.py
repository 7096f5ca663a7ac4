"""GPU parity at the library's maximum sizes: capacity GEAR_MAX_CAPACITY
(2^30 slots, selection-only table) and batch GEAR_MAX_BATCH (2^24 draws).
Inputs are seeded numpy draws (uniform, with zeros), compared with the
oracle on the same arrays."""
import numpy as np
import pytest
import torch

import oracle
from paper_2310_05205_amd import gear
from tests.helpers import DEV, assert_weights, cuda, host, say

pytestmark = pytest.mark.gpu


def _table(p, T=1):
    t = gear.Table([], p.size, T, gear.GEAR_DEVICE, DEV)
    t.insert([], p)
    return t


def test_max_capacity_prioritized_and_topk():
    N = gear.GEAR_MAX_CAPACITY
    rng = np.random.default_rng(30)
    say("max capacity: generating %d priorities" % N)
    p = rng.integers(0, 1 << 24, size=N, dtype=np.uint32)
    p[rng.integers(0, N, size=N // 8)] = 0
    t = _table(p)
    try:
        for it, (B, beta) in enumerate([(8192, 0.4), (100000, 1.0)]):
            say("max capacity prioritized B=%d" % B)
            seed = 0x5EED0000 + it
            st, oidx, ostart, ow = oracle.select(oracle.PRIORITIZED, p, N, 1, B, 1, seed, beta, True)
            idx, start, w = t.select(gear.GEAR_PRIORITIZED, B, 1, seed, beta, weights=True)
            np.testing.assert_array_equal(host(idx), oidx)
            assert_weights(host(w), ow)
        assert t.sync() == 0
        # TopK over the same 2^30 slots after most priorities are cleared:
        # the candidates are few enough for the oracle's sort.
        keep = rng.integers(0, N, size=2_000_000)
        q = np.zeros(N, dtype=np.uint32)
        q[keep] = p[keep]
        t.close()
        t = _table(q)
        for K in (16384, 777):
            say("max capacity TopK K=%d" % K)
            st, oidx, _, _ = oracle.select(oracle.TOPK, q, N, 1, K, 1, 3, 0.0, False)
            idx, _, _ = t.select(gear.GEAR_TOPK, K, 1, 3)
            np.testing.assert_array_equal(host(idx), oidx)
        assert t.sync() == 0
    finally:
        t.close()


def test_max_batch_select_collect_update():
    B = gear.GEAR_MAX_BATCH
    N, T, L = 1 << 22, 3, 1
    rng = np.random.default_rng(24)
    p = rng.integers(1, 1 << 20, size=N, dtype=np.uint32)
    col = rng.integers(0, 256, size=(N, T * 4), dtype=np.uint8)
    t = gear.Table([4], N, T, gear.GEAR_DEVICE, DEV)
    try:
        t.insert([col], p)
        say("max batch: prioritized select of %d draws" % B)
        st, oidx, ostart, ow = oracle.select(oracle.PRIORITIZED, p, N, T, B, L, 2424, 0.4, True)
        idx, start, w = t.select(gear.GEAR_PRIORITIZED, B, L, 2424, 0.4, weights=True)
        np.testing.assert_array_equal(host(idx), oidx)
        np.testing.assert_array_equal(host(start), ostart)
        assert_weights(host(w), ow)
        say("max batch: collect")
        out = host(t.collect(idx, start, L)[0]).reshape(B, 4)
        sample = rng.integers(0, B, size=100000)
        np.testing.assert_array_equal(out[sample], col.reshape(N, T, 4)[oidx[sample], ostart[sample]])
        say("max batch: update (tag path)")
        newp = rng.integers(1, 1 << 20, size=B, dtype=np.uint32)
        t.update_priorities(idx, torch.from_numpy(newp).to(cuda()))
        assert oracle.update(p, oidx, newp) == oracle.OK
        torch.cuda.synchronize(DEV)
        np.testing.assert_array_equal(t.priorities(), p)
        assert t.sync() == 0
    finally:
        t.close()
