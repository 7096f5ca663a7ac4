"""gear_select_collect: FIFO, LIFO and uniform selection and the gather of
their windows in one launch, against the oracle and against gear_select
followed by gear_collect (the same slots, starts, weights and bytes).

The fused kernel computes each window's slot and start itself and writes the
draws from the piece that holds each window's first element, so the cases
cover wide and narrow columns, whole trajectories (16-byte elements), pieces
that span two windows, partial and wrapped rings, index-manager tables (draws
over the commit order), more columns than one launch takes, and pinned host
tables."""
import dataclasses

import numpy as np
import pytest

import gen
import oracle
from gen import configs
from paper_2310_05205_amd import gear
from tests.helpers import gpu_table, host, oracle_priorities, oracle_windows, say
from tests.test_parity_gpu import ODD, RANDOM, U1000, _custom

pytestmark = pytest.mark.gpu

SIMPLE = (gear.GEAR_FIFO, gear.GEAR_LIFO, gear.GEAR_UNIFORM)


def _two_call(t, strategy, B, L, seed, col_ids=None):
    idx, start, w = t.select(strategy, B, L, seed, 0.0, weights=True)
    return idx, start, w, t.collect(idx, start, L, col_ids=col_ids)


def _assert_same(a, b, what):
    for x, y, name in zip(a[:3], b[:3], ("idx", "start", "weights")):
        np.testing.assert_array_equal(host(x), host(y), err_msg="%s: %s" % (what, name))
    assert len(a[3]) == len(b[3])
    for c, (x, y) in enumerate(zip(a[3], b[3])):
        np.testing.assert_array_equal(host(x), host(y), err_msg="%s: column %d" % (what, c))


def _against_oracle(w, t, p, next_seq, strategy, B, L, seed):
    """The fused call's draws against the oracle's ring arithmetic, and every
    gathered window against the oracle's collection of the selected
    trajectories (regenerated on the CPU)."""
    got = t.select_collect(strategy, B, L, seed, weights=True)
    st, oidx, ostart, ow = oracle.select(strategy, p, next_seq, w.T, B, L, seed, 0.0, True)
    assert st == oracle.OK
    np.testing.assert_array_equal(host(got[0]), oidx)
    np.testing.assert_array_equal(host(got[1]), ostart)
    np.testing.assert_array_equal(host(got[2]), ow)
    ref = oracle_windows(w, oidx, ostart, L, next_seq, np.arange(B))
    for c in range(len(w.columns)):
        np.testing.assert_array_equal(host(got[3][c]), ref[c], err_msg="%s column %d" % (w.name, c))
    return got


CASES = [
    configs.DT,                                                       # wrapped ring, 20-step windows
    dataclasses.replace(configs.DT, name="dt-whole", L=configs.DT.T),  # whole trajectories, 16-byte elements
    configs.TINY,
    _custom("partial-fill", 4097, 3, ODD[:3], 700, U1000, 64, 1, strategies=SIMPLE),
    _custom("wrapped", 300, 4, ODD[:4], 1234, U1000, 100, 2, strategies=SIMPLE),
    _custom("wide-narrow-mix", 2000, 40, ODD, 2000, U1000, 700, 33, strategies=SIMPLE),
    _custom("batch-one", 777, 6, ODD[:3], 777, U1000, 1, 6, strategies=SIMPLE),
    _custom("full-window-16B", 3000, 4, ODD[2:4], 3000, U1000, 500, 4, strategies=SIMPLE),
    _custom("one-slot", 1, 5, ODD[:2], 1, U1000, 1, 5, strategies=SIMPLE),
]


@pytest.mark.parametrize("w", CASES, ids=[w.name for w in CASES])
def test_select_collect_matches_oracle_and_two_calls(w):
    p, next_seq = oracle_priorities(w)
    t = gpu_table(w)
    try:
        for it in range(2):
            seed = gen.select_seed(w.seed, it)
            for strategy in SIMPLE:
                say("%s select_collect iteration %d strategy %d" % (w.name, it, strategy))
                B = w.B if strategy == gear.GEAR_UNIFORM else min(w.B, min(w.n_insert, w.N))
                got = _against_oracle(w, t, p, next_seq, strategy, B, w.L, seed)
                _assert_same(got, _two_call(t, strategy, B, w.L, seed), w.name)
                del got
        assert t.sync() == 0
    finally:
        t.close()


SIMPLE_RANDOM = [w for w in RANDOM if w.columns and any(st in SIMPLE for st in w.strategies)]


@pytest.mark.parametrize("w", SIMPLE_RANDOM, ids=[w.name for w in SIMPLE_RANDOM])
def test_select_collect_random_configurations(w):
    t = gpu_table(w)
    try:
        live = min(w.n_insert, w.N)
        for strategy in (st for st in w.strategies if st in SIMPLE):
            seed = gen.select_seed(w.seed, 3)
            B = w.B if strategy == gear.GEAR_UNIFORM else min(w.B, live)
            say("%s select_collect strategy %d B=%d L=%d" % (w.name, strategy, B, w.L))
            _assert_same(t.select_collect(strategy, B, w.L, seed, weights=True),
                         _two_call(t, strategy, B, w.L, seed), w.name)
        assert t.sync() == 0
    finally:
        t.close()


def test_select_collect_column_subsets_and_many_columns():
    """Columns requested in another order, a subset, and 20 columns (two
    launches: only the first writes the draws)."""
    cols = [ODD[k % len(ODD)] for k in range(20)]
    w = _custom("twenty-columns", 500, 12, cols, 700, U1000, 300, 7, strategies=SIMPLE)
    t = gpu_table(w)
    try:
        for ids in ([5, 3, 0], [1], None):
            for strategy in SIMPLE:
                seed = gen.select_seed(w.seed, 1)
                say("twenty-columns select_collect col_ids %s strategy %d" % (ids, strategy))
                _assert_same(t.select_collect(strategy, w.B, w.L, seed, weights=True, col_ids=ids),
                             _two_call(t, strategy, w.B, w.L, seed, col_ids=ids), "twenty-columns")
        assert t.sync() == 0
    finally:
        t.close()


@pytest.mark.parametrize("removal", [gear.GEAR_FIFO, gear.GEAR_LIFO], ids=["fifo", "lifo"])
def test_select_collect_over_the_commit_order(removal):
    """A table with an index manager: the draws are positions in the commit
    order, read from the device's commit-order ring."""
    N, T, E = 200, 6, [8, 3]
    t = gear.Table(E, N, T, gear.GEAR_DEVICE, 0)
    rng = np.random.default_rng(5)
    try:
        t.use_allocator(removal, 150)
        for step in range(4):
            n = int(rng.integers(40, 90))
            rows = [rng.integers(0, 256, (n, T * e), dtype=np.uint8) for e in E]
            t.insert(rows, rng.integers(1, 1000, n).astype(np.uint32))
            for strategy in SIMPLE:
                seed = 1000 + step
                say("commit order step %d strategy %d" % (step, strategy))
                _assert_same(t.select_collect(strategy, 32, 3, seed, weights=True),
                             _two_call(t, strategy, 32, 3, seed), "commit order")
        assert t.sync() == 0
    finally:
        t.close()


def test_select_collect_pinned_host_table():
    w = dataclasses.replace(_custom("host", 3000, 5, ODD[1:5], 4500, U1000, 333, 3, strategies=SIMPLE),
                            host_table=True)
    p, next_seq = oracle_priorities(w)
    t = gpu_table(w)
    try:
        for strategy in SIMPLE:
            say("pinned host select_collect strategy %d" % strategy)
            _against_oracle(w, t, p, next_seq, strategy, w.B, w.L, gen.select_seed(w.seed, 0))
        assert t.sync() == 0
    finally:
        t.close()


def test_select_collect_errors():
    t = gear.Table([4], 10, 3, gear.GEAR_DEVICE, 0)
    try:
        with pytest.raises(gear.GearError) as e:
            t.select_collect(gear.GEAR_UNIFORM, 4, 2, 1)
        assert e.value.code == gear.GEAR_E_EMPTY
        t.insert([np.zeros((5, 12), np.uint8)], np.ones(5, dtype=np.uint32))
        with pytest.raises(gear.GearError) as e:
            t.select_collect(gear.GEAR_FIFO, 6, 2, 1)
        assert e.value.code == gear.GEAR_E_INSUFFICIENT
        for strategy in (gear.GEAR_PRIORITIZED, gear.GEAR_TOPK, 9):
            with pytest.raises(gear.GearError) as e:
                t.select_collect(strategy, 2, 2, 1)
            assert e.value.code == gear.GEAR_E_INVAL
        with pytest.raises(gear.GearError) as e:
            t.select_collect(gear.GEAR_UNIFORM, 2, 4, 1)  # L > T
        assert e.value.code == gear.GEAR_E_INVAL
        idx, start, w, outs = t.select_collect(gear.GEAR_LIFO, 5, 3, 1, weights=True)
        np.testing.assert_array_equal(host(idx), [4, 3, 2, 1, 0])
        assert t.sync() == 0
    finally:
        t.close()
