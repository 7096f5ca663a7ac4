"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Integer outputs (indices, window starts, gathered bytes, priorities after an
update) must be bit-identical; importance-sampling weights agree within
1e-6 relative (fp64 arithmetic on both sides, rounded once to fp32).
"""
import dataclasses

import numpy as np
import pytest
import torch

import gen
import oracle
from gen import configs
from paper_2310_05205_amd import gear
from tests.helpers import (assert_weights, cuda, gpu_table, host, oracle_priorities, oracle_store,
                           oracle_windows, say)

pytestmark = pytest.mark.gpu

KINDS = [
    gen.Column("bytes", gen.BYTES, 12288), gen.Column("bytes_odd", gen.BYTES, 3),
    gen.Column("nf32", gen.NORMAL_F32, 17), gen.Column("uf32", gen.UNIFORM_F32, 6),
    gen.Column("int", gen.INT_MOD, 8, param=16), gen.Column("bf16", gen.NORMAL_BF16, 512),
    gen.Column("done", gen.DONE_U8, 1), gen.Column("rtg", gen.RTG_F32, 1, param=2),
    gen.Column("stamp", gen.STAMP, 1),
]


@pytest.mark.parametrize("col", KINDS, ids=[c.name for c in KINDS])
def test_generator_gpu_matches_cpu(col):
    say("generator twin %s" % col.name)
    T, k0, n = 37, 1000, 5
    d = torch.empty(n * T * col.elem_bytes, dtype=torch.uint8, device=cuda())
    gen.fill_rows_gpu(col, 3, 77, T, k0, n, d.data_ptr(), torch.cuda.current_stream().cuda_stream)
    np.testing.assert_array_equal(host(d).reshape(n, -1), gen.fill_rows_cpu(col, 3, 77, T, k0, n))


def _check_table_contents(t, w, s):
    """Every column of the HIP table equals the oracle store's."""
    for c in range(len(w.columns)):
        base, hptr, eb = gear.gear_table_column(t.handle, c)
        nbytes = w.N * w.T * eb
        if hptr:
            got = np.ctypeslib.as_array((np.ctypeslib.ctypes.c_uint8 * nbytes).from_address(hptr))
        else:
            got = np.empty(nbytes, dtype=np.uint8)
            gear._hip_memcpy_d2h(got.ctypes.data, base, nbytes)
        np.testing.assert_array_equal(got.reshape(w.N, -1), s.cols[c])
    np.testing.assert_array_equal(t.priorities(), s.priority)


def _run_full(w, iterations, strategies=None, check_contents=True, options=0):
    """Full comparison on a workload small enough for a full oracle store."""
    s = oracle_store(w)
    t = gpu_table(w, options=options)
    try:
        if check_contents:
            _check_table_contents(t, w, s)
        for it in range(iterations):
            seed = gen.select_seed(w.seed, it)
            for strat in (strategies or w.strategies):
                say("%s iteration %d strategy %d" % (w.name, it, strat))
                B = w.B
                idx, start, wt = t.select(strat, B, w.L, seed, w.beta, weights=w.weights)
                st, oidx, ostart, ow = s.select(strat, B, w.L, seed, w.beta, weights=w.weights,
                                                global_min=bool(options & gear.GEAR_OPT_IS_GLOBAL_MIN))
                assert st == oracle.OK
                np.testing.assert_array_equal(host(idx), oidx)
                np.testing.assert_array_equal(host(start), ostart)
                if w.weights:
                    assert_weights(host(wt), ow)
                if w.columns:
                    outs = t.collect(idx, start, w.L)
                    st, oouts = s.collect(oidx, ostart, w.L)
                    assert st == oracle.OK
                    for c in range(len(w.columns)):
                        np.testing.assert_array_equal(host(outs[c]), oouts[c])
                if strat == gear.GEAR_PRIORITIZED:
                    newp = gen.update_priorities(w.prio, w.seed, it, B)
                    t.update_priorities(idx, torch.from_numpy(newp).to(cuda()))
                    assert s.update(oidx, newp) == oracle.OK
                    np.testing.assert_array_equal(t.priorities(), s.priority)
        assert t.sync() == 0
    finally:
        t.close()


def test_tiny_prioritized_replay():
    _run_full(configs.TINY, iterations=5)


@pytest.mark.parametrize("options", [0, gear.GEAR_OPT_INCREMENTAL_TREE], ids=["rescan", "incremental"])
def test_selection_stress_100_iterations(options):
    w = configs.SELECT_STRESS
    p, next_seq = oracle_priorities(w)
    t = gpu_table(w, options=options)
    try:
        np.testing.assert_array_equal(t.priorities(), p)
        for it in range(w.iterations):
            say("selection stress iteration %d" % it)
            seed = gen.select_seed(w.seed, it)
            idx, start, wt = t.select(gear.GEAR_PRIORITIZED, w.B, w.L, seed, w.beta, weights=True)
            st, oidx, ostart, ow = oracle.select(oracle.PRIORITIZED, p, next_seq, w.T, w.B, w.L, seed, w.beta, True)
            assert st == oracle.OK
            np.testing.assert_array_equal(host(idx), oidx)
            np.testing.assert_array_equal(host(start), ostart)
            assert_weights(host(wt), ow)
            newp = gen.update_priorities(w.prio, w.seed, it, w.B)
            t.update_priorities(idx, torch.from_numpy(newp).to(cuda()))
            assert oracle.update(p, oidx, newp) == oracle.OK
            np.testing.assert_array_equal(t.priorities(), p)
        assert t.sync() == 0
    finally:
        t.close()


def test_dt_uniform_fifo_lifo_wrapped_ring():
    w = configs.DT
    t = gpu_table(w)
    try:
        count, next_seq = t.info()
        assert (count, next_seq) == (w.N, w.n_insert)
        zeros = np.zeros(w.N, dtype=np.uint32)
        for strat in w.strategies:
            say("dt strategy %d" % strat)
            seed = gen.select_seed(w.seed, 0)
            idx, start, _ = t.select(strat, w.B, w.L, seed)
            st, oidx, ostart, _ = oracle.select(strat, zeros, next_seq, w.T, w.B, w.L, seed)
            assert st == oracle.OK
            np.testing.assert_array_equal(host(idx), oidx)
            np.testing.assert_array_equal(host(start), ostart)
            outs = t.collect(idx, start, w.L)
            ref = oracle_windows(w, oidx, ostart, w.L, next_seq, np.arange(w.B))
            for c in range(len(w.columns)):
                np.testing.assert_array_equal(host(outs[c]), ref[c])
        # Full-trajectory windows (L = T) of the newest 64 insertions.
        idx, start, _ = t.select(gear.GEAR_LIFO, 64, w.T, 1)
        outs = t.collect(idx, start, w.T)
        st, oidx, ostart, _ = oracle.select(oracle.LIFO, zeros, next_seq, w.T, 64, w.T, 1)
        ref = oracle_windows(w, oidx, ostart, w.T, next_seq, np.arange(64))
        for c in range(len(w.columns)):
            np.testing.assert_array_equal(host(outs[c]), ref[c])
        assert t.sync() == 0
    finally:
        t.close()


def test_dt_full_trajectories():
    # The bench's full-trajectory workload: 512 whole trajectories (L = T =
    # 1000) by each strategy, every window against the oracle.
    w = configs.DT_FULL
    t = gpu_table(w)
    try:
        _, next_seq = t.info()
        zeros = np.zeros(w.N, dtype=np.uint32)
        for strat in w.strategies:
            say("dt-full strategy %d" % strat)
            seed = gen.select_seed(w.seed, 7)
            idx, start, _ = t.select(strat, w.B, w.L, seed)
            st, oidx, ostart, _ = oracle.select(strat, zeros, next_seq, w.T, w.B, w.L, seed)
            assert st == oracle.OK
            np.testing.assert_array_equal(host(idx), oidx)
            assert not np.any(host(start))
            outs = t.collect(idx, start, w.L)
            ref = oracle_windows(w, oidx, ostart, w.L, next_seq, np.arange(w.B))
            for c in range(len(w.columns)):
                np.testing.assert_array_equal(host(outs[c]), ref[c])
        assert t.sync() == 0
    finally:
        t.close()


# ---------------------------------------------------------------------------
# Edge cases: ragged tails, tiny and multi-level prefix trees, odd element
# sizes, partial fills, wrap-around, zero runs and large priorities.
# ---------------------------------------------------------------------------

def _custom(name, N, T, cols, n_insert, prio, B, L, strategies=(3,), weights=True, seed=11):
    return configs.Workload(name=name, seed=seed, N=N, T=T, columns=tuple(cols), n_insert=n_insert, prio=prio,
                            strategies=tuple(strategies), B=B, L=L, weights=weights)


U1000 = gen.PrioDist(gen.PRIO_UNIFORM, 1, 1000)
BIG = gen.PrioDist(gen.PRIO_UNIFORM, 0xF0000000, 0xFFFFFFFF)
SPARSE = gen.PrioDist(gen.PRIO_PARETO, 0.3, float(0xFFFFFFFF))
ODD = [gen.Column("b1", gen.DONE_U8, 1), gen.Column("b3", gen.BYTES, 3), gen.Column("w12", gen.INT_MOD, 3, param=7),
       gen.Column("w68", gen.NORMAL_F32, 17), gen.Column("v32", gen.INT_MOD, 8, param=16),
       gen.Column("v1024", gen.NORMAL_BF16, 512)]

EDGE = [
    _custom("one-slot", 1, 5, ODD[:2], 1, U1000, 7, 5),
    _custom("ragged-1000", 1000, 9, ODD, 1000, U1000, 333, 4),
    _custom("partial-fill", 4097, 3, ODD[:3], 700, U1000, 64, 1, strategies=(0, 1, 2, 3)),
    _custom("wrapped", 300, 4, ODD[:4], 1234, U1000, 100, 2, strategies=(0, 1, 2, 3)),
    _custom("big-priorities", 5000, 2, ODD[3:5], 5000, BIG, 2048, 2),
    _custom("heavy-tail", 20000, 1, [], 20000, SPARSE, 4096, 1),
    _custom("lookback-depth", 300000, 1, [], 300000, U1000, 1024, 1),
    _custom("two-levels", (1 << 22) + 17, 1, [], (1 << 22) + 17, U1000, 4096, 1),
    _custom("three-levels", (1 << 24) + 5, 1, [], (1 << 24) + 5, U1000, 4096, 1),
    _custom("wide-level1", (1 << 26) + 4097, 1, [], (1 << 26) + 4097, U1000, 4096, 1),
    _custom("big-batch", 300000, 1, [], 300000, U1000, 12000, 1),
    _custom("wide-narrow-mix", 2000, 40, ODD, 2000, U1000, 700, 33),
    _custom("batch-one", 777, 6, ODD[:3], 777, U1000, 1, 6),
    # L = T with step sizes of 12 and 68 bytes: every window starts at step
    # 0, 48 and 272 bytes apart, so the 16-byte path applies.
    _custom("full-window-16B", 3000, 4, ODD[2:4], 3000, U1000, 500, 4),
]


@pytest.mark.parametrize("options", [0, gear.GEAR_OPT_INCREMENTAL_TREE], ids=["rescan", "incremental"])
@pytest.mark.parametrize("w", EDGE, ids=[w.name for w in EDGE])
def test_edge_cases(w, options):
    big = w.N > 100000
    if big:
        # Selection-only shapes: compare without a full oracle store.
        p, next_seq = oracle_priorities(w)
        t = gpu_table(w, options=options)
        try:
            for it in range(3):
                say("%s iteration %d" % (w.name, it))
                seed = gen.select_seed(w.seed, it)
                idx, start, wt = t.select(3, w.B, w.L, seed, w.beta, weights=True)
                st, oidx, ostart, ow = oracle.select(3, p, next_seq, w.T, w.B, w.L, seed, w.beta, True)
                assert st == oracle.OK
                np.testing.assert_array_equal(host(idx), oidx)
                assert_weights(host(wt), ow)
                newp = gen.update_priorities(w.prio, w.seed, it, w.B)
                t.update_priorities(idx, torch.from_numpy(newp).to(cuda()))
                oracle.update(p, oidx, newp)
                np.testing.assert_array_equal(t.priorities(), p)
        finally:
            t.close()
    else:
        _run_full(w, iterations=3, options=options)


def test_more_than_sixteen_columns_and_subsets():
    cols = [gen.Column("c%d" % i, gen.INT_MOD, 1 + (i % 5), param=1000 + i) for i in range(20)]
    w = _custom("twenty-columns", 500, 12, cols, 500, U1000, 300, 7)
    s = oracle_store(w)
    t = gpu_table(w)
    try:
        idx, start, _ = t.select(3, w.B, w.L, 5)
        st, oidx, ostart, _ = s.select(3, w.B, w.L, 5)
        np.testing.assert_array_equal(host(idx), oidx)
        outs = t.collect(idx, start, w.L)
        _, ref = s.collect(oidx, ostart, w.L)
        for c in range(20):
            np.testing.assert_array_equal(host(outs[c]), ref[c])
        sub = [17, 3, 3, 0]
        outs = t.collect(idx, start, w.L, col_ids=sub)
        _, ref = s.collect(oidx, ostart, w.L, col_ids=sub)
        for j in range(len(sub)):
            np.testing.assert_array_equal(host(outs[j]), ref[j])
    finally:
        t.close()


@pytest.mark.parametrize("options", [0, gear.GEAR_OPT_INCREMENTAL_TREE], ids=["rescan", "incremental"])
@pytest.mark.parametrize("B", [1, 5000, 8192, 8193, 20000])
def test_duplicate_heavy_update_last_wins(B, options):
    # B <= 8192 runs the one-launch LDS path, larger B the two-kernel path.
    w = _custom("dups", 100, 1, [], 100, U1000, B, 1)
    p, next_seq = oracle_priorities(w)
    t = gpu_table(w, options=options)
    t.select(3, 16, 1, 1)   # builds the tree, so updates maintain it when asked
    try:
        rng = np.random.default_rng(B)
        for it in range(5):
            say("dups B=%d iteration %d" % (B, it))
            idx = rng.integers(0, w.N, size=B)
            newp = rng.integers(1, 1 << 32, size=B, dtype=np.uint64).astype(np.uint32)
            t.update_priorities(torch.from_numpy(idx).to(cuda()), torch.from_numpy(newp).to(cuda()))
            oracle.update(p, idx, newp)
            np.testing.assert_array_equal(t.priorities(), p)
            sel, _, _ = t.select(3, 4096, 1, 100 + it)
            _, osel, _, _ = oracle.select(3, p, next_seq, 1, 4096, 1, 100 + it)
            np.testing.assert_array_equal(host(sel), osel)
        assert t.sync() == 0
    finally:
        t.close()


def test_insert_longer_than_capacity_keeps_last_rows():
    w = _custom("overfull", 64, 3, [gen.Column("stamp", gen.STAMP, 1)], 200, U1000, 16, 3, strategies=(0, 1))
    s = oracle.Store(w.elem_bytes, w.N, w.T)
    rows = gen.fill_rows_cpu(w.columns[0], 0, w.seed, w.T, 0, w.n_insert)
    prio = gen.insert_priorities(w.prio, w.seed, 0, w.n_insert)
    s.insert([rows], prio)
    t = gear.Table(w.elem_bytes, w.N, w.T)
    try:
        t.insert([rows], prio)           # host sources, one call with n > N
        _check_table_contents(t, w, s)
        for strat in (0, 1):
            idx, start, _ = t.select(strat, w.N, 2, 9)
            _, oidx, ostart, _ = s.select(strat, w.N, 2, 9)
            np.testing.assert_array_equal(host(idx), oidx)
    finally:
        t.close()


def test_pinned_host_table_small():
    w = dataclasses.replace(configs.TINY, host_table=True, name="tiny-pinned")
    _run_full(w, iterations=2)


def test_cdf_reuse_and_rescan():
    w = _custom("reuse", 3000, 1, [], 3000, U1000, 500, 1)
    p, next_seq = oracle_priorities(w)
    t = gpu_table(w)
    try:
        a, _, _ = t.select(3, w.B, 1, 42)
        b, _, _ = t.select(3, w.B, 1, 42)           # no change: scan reused
        np.testing.assert_array_equal(host(a), host(b))
        newp = np.full(w.B, 7, dtype=np.uint32)
        t.update_priorities(a, torch.from_numpy(newp).to(cuda()))
        oracle.update(p, host(a), newp)
        c, _, _ = t.select(3, w.B, 1, 42)           # changed: rescanned
        _, oc, _, _ = oracle.select(3, p, next_seq, 1, w.B, 1, 42)
        np.testing.assert_array_equal(host(c), oc)
    finally:
        t.close()


def test_device_status_and_host_errors():
    t = gear.Table([4, 1], 10, 8)
    try:
        idx = torch.zeros(4, dtype=torch.int64, device=cuda())
        with pytest.raises(gear.GearError) as e:
            t.select(2, 4, 2, 0)
        assert e.value.code == gear.GEAR_E_EMPTY
        rows = [np.zeros((3, 32), np.uint8), np.zeros((3, 8), np.uint8)]
        t.insert(rows, np.zeros(3, dtype=np.uint32))              # all priorities zero
        with pytest.raises(gear.GearError) as e:
            t.select(0, 4, 2, 0)
        assert e.value.code == gear.GEAR_E_INSUFFICIENT
        with pytest.raises(gear.GearError) as e:
            t.select(3, 4, 9, 0)
        assert e.value.code == gear.GEAR_E_INVAL
        idx, start, wt = t.select(3, 4, 2, 0, 0.4, weights=True)
        assert np.all(host(idx) == -1) and np.all(host(start) == 0) and np.all(host(wt) == 0)
        assert t.sync() == gear.GEAR_STATUS_NO_WEIGHT
        assert t.sync() == 0
        bad = torch.tensor([0, 10, -1, 2], dtype=torch.int64, device=cuda())
        st = torch.tensor([0, 0, 0, 7], dtype=torch.int32, device=cuda())
        outs = t.collect(bad, st, 2)
        assert np.all(host(outs[0])[1:] == 0) and np.all(host(outs[1])[1:] == 0)
        assert t.sync() == gear.GEAR_STATUS_BAD_INDEX
        t.update_priorities(torch.tensor([5, 1], dtype=torch.int64, device=cuda()),
                            torch.tensor([9, 9], dtype=torch.int32, device=cuda()))
        assert t.sync() == gear.GEAR_STATUS_BAD_INDEX         # slot 5 is not live
        np.testing.assert_array_equal(t.priorities()[:3], [0, 9, 0])
    finally:
        t.close()


# ---------------------------------------------------------------------------
# Full-size workloads, in the launch configuration the benchmark times.
# ---------------------------------------------------------------------------

def _full_size(w, iterations, sample_n, options=0):
    """Every iteration compares all draws and weights; the first compares
    every gathered window of the batch (the oracle regenerates all B selected
    trajectories), later ones sample_n windows including the first and last."""
    p, next_seq = oracle_priorities(w)
    t = gpu_table(w, options=options)
    rng = np.random.default_rng(w.seed)
    try:
        for it in range(iterations):
            say("%s iteration %d" % (w.name, it))
            seed = gen.select_seed(w.seed, it)
            idx, start, wt = t.select(3, w.B, w.L, seed, w.beta, weights=True)
            outs = t.collect(idx, start, w.L)
            st, oidx, ostart, ow = oracle.select(3, p, next_seq, w.T, w.B, w.L, seed, w.beta, True)
            assert st == oracle.OK
            np.testing.assert_array_equal(host(idx), oidx)
            np.testing.assert_array_equal(host(start), ostart)
            assert_weights(host(wt), ow)
            if it == 0:
                sample = np.arange(w.B)
            else:
                sample = np.sort(rng.choice(w.B, size=sample_n, replace=False))
                sample[0], sample[-1] = 0, w.B - 1
            ref = oracle_windows(w, oidx, ostart, w.L, next_seq, sample)
            for c in range(len(w.columns)):
                got = host(outs[c]) if it == 0 else host(outs[c][torch.from_numpy(sample).to(cuda())])
                np.testing.assert_array_equal(got, ref[c])
            del outs, ref, got
            newp = gen.update_priorities(w.prio, w.seed, it, w.B)
            t.update_priorities(idx, torch.from_numpy(newp).to(cuda()))
            oracle.update(p, oidx, newp)
            np.testing.assert_array_equal(t.priorities(), p)
        assert t.sync() == 0
    finally:
        t.close()


def test_gato_pinned_host_zero_copy_full_size():
    _full_size(configs.GATO_HOST, iterations=2, sample_n=64)


@pytest.mark.parametrize("options", [0, gear.GEAR_OPT_INCREMENTAL_TREE], ids=["rescan", "incremental"])
def test_mat_end_to_end_full_size(options):
    _full_size(configs.MAT, iterations=3, sample_n=256, options=options)


# ---------------------------------------------------------------------------
# TopK selection (deterministic: highest priorities, lower slot on ties).
# ---------------------------------------------------------------------------

TOPK_CASES = [
    _custom("topk-one", 1, 3, [], 1, U1000, 1, 2, strategies=(4,)),
    _custom("topk-ties", 1000, 3, [], 1000, gen.PrioDist(gen.PRIO_UNIFORM, 1, 3), 777, 2, strategies=(4,)),
    _custom("topk-short", 4097, 2, [], 300, U1000, 1024, 1, strategies=(4,)),       # 300 live < K
    _custom("topk-big-values", 100000, 1, [], 100000, BIG, 5000, 1, strategies=(4,)),
    _custom("topk-heavy-tail", 300000, 1, [], 300000, SPARSE, 16384, 1, strategies=(4,)),
    _custom("topk-pareto-4M", 1 << 22, 1, [], 1 << 22, gen.PrioDist(gen.PRIO_PARETO, 1.5, float(1 << 24)), 8192, 1,
            strategies=(4,)),
    # 4096 large values sharing their top 24 key bits: all three digit passes run.
    _custom("topk-three-pass", 100000, 1, [], 100000, gen.PrioDist(gen.PRIO_UNIFORM, 0x80000000, 0x80000FFF), 5000, 1,
            strategies=(4,)),
    # Several batches per workgroup with a ragged tail, and the largest K.
    _custom("topk-multi-batch-maxK", (1 << 23) + 12345, 1, [], (1 << 23) + 12345,
            gen.PrioDist(gen.PRIO_LOGNORMAL, 6.931471805599453, 1.0, float(1 << 24)), 16384, 1, strategies=(4,)),
]


@pytest.mark.parametrize("w", TOPK_CASES, ids=[w.name for w in TOPK_CASES])
def test_topk_matches_oracle(w):
    p, next_seq = oracle_priorities(w)
    t = gpu_table(w)
    try:
        for it in range(3):
            say("%s iteration %d" % (w.name, it))
            seed = gen.select_seed(w.seed, it)
            idx, start, wt = t.select(gear.GEAR_TOPK, w.B, w.L, seed, 0.0, weights=True)
            st, oidx, ostart, ow = oracle.select(oracle.TOPK, p, next_seq, w.T, w.B, w.L, seed, 0.0, True)
            np.testing.assert_array_equal(host(idx), oidx)
            np.testing.assert_array_equal(host(start), ostart)
            np.testing.assert_array_equal(host(wt), ow)
            assert t.sync() == (0 if st == oracle.OK else gear.GEAR_STATUS_NO_WEIGHT)
            # New priorities for the selected slots change the next TopK.
            sel = oidx[oidx >= 0]
            newp = gen.update_priorities(w.prio, w.seed, it, sel.size) // 2
            t.update_priorities(torch.from_numpy(sel).to(cuda()), torch.from_numpy(newp).to(cuda()))
            oracle.update(p, sel, newp)
    finally:
        t.close()


def test_topk_rejects_oversized_batch():
    t = gear.Table([4], 10, 2)
    try:
        t.insert([np.zeros((10, 8), np.uint8)], np.ones(10, dtype=np.uint32))
        with pytest.raises(gear.GearError) as e:
            t.select(gear.GEAR_TOPK, gear.GEAR_MAX_TOPK + 1, 1, 0)
        assert e.value.code == gear.GEAR_E_INVAL
    finally:
        t.close()


def _boundary_priorities(rng, N):
    """Priorities clustered around powers of two (2^e - 2 .. 2^e + 2 for
    several e, and the top of the 32-bit range), where the TopK threshold's
    digit prefix changes leading-one position, plus uniform filler.  Returns
    the priorities and the cluster values."""
    centres = [1 << e for e in (1, 2, 7, 8, 9, 12, 20, 24, 31)]
    cluster = np.array(sorted({c + d for c in centres for d in (-2, -1, 0, 1, 2)} |
                              {1, 2, 3, 0xFFFFFFFE, 0xFFFFFFFF}), dtype=np.uint64)
    p = np.where(rng.random(N) < 0.7, cluster[rng.integers(0, cluster.size, N)],
                 rng.integers(1, 1 << 32, N, dtype=np.uint64))
    p[rng.random(N) < 0.05] = 0
    return p.astype(np.uint32), cluster.astype(np.uint32)


def test_topk_threshold_at_exponent_boundaries():
    """The K-th largest priority placed at and next to powers of two: K is
    each cluster value's first and last position in descending order, so the
    threshold falls on every side of every boundary."""
    rng = np.random.default_rng(20)
    N, T = 12000, 2  # every non-zero priority lies within the first GEAR_MAX_TOPK places
    p, cluster = _boundary_priorities(rng, N)
    t = gear.Table([1], capacity=N, T=T, residency=gear.GEAR_DEVICE, device=0)
    try:
        t.insert([np.zeros((N, T), np.uint8)], p)
        order = np.argsort(-p.astype(np.int64), kind="stable")
        desc = p[order]
        ks = set()
        for v in cluster:
            pos = np.nonzero(desc == v)[0]
            if pos.size == 0:
                continue
            ks.update({int(pos[0]) + 1, int(pos[-1]) + 1, int(pos[-1]) + 2})
        ks = sorted(k for k in ks if 1 <= k <= gear.GEAR_MAX_TOPK)
        say("TopK at %d thresholds around powers of two" % len(ks))
        for K in ks:
            idx, start, wt = t.select(gear.GEAR_TOPK, K, 1, 7, 0.0, weights=True)
            st, oidx, ostart, ow = oracle.select(oracle.TOPK, p, N, T, K, 1, 7, 0.0, True)
            np.testing.assert_array_equal(host(idx), oidx, err_msg="K=%d" % K)
            np.testing.assert_array_equal(host(start), ostart)
            np.testing.assert_array_equal(host(wt), ow)
            assert t.sync() == (0 if st == oracle.OK else gear.GEAR_STATUS_NO_WEIGHT)
    finally:
        t.close()


def test_topk_threshold_bin_taken_whole():
    """K ends exactly at the end of a digit bin that holds many distinct
    priorities, so the threshold is a range of values, not one value: the
    keys at it are in slot order but not in priority order and must be
    ranked by comparison.  A bin of the first digit pass (from 2^20: 8192
    values per bin), and one of the second (from 2^28 + 2^20: 512 values per
    bin) whose first-pass bin also holds lower keys, so the first pass does
    not decide."""
    rng = np.random.default_rng(21)
    N, T, M = 60000, 2, 3000
    for base, width, lower in ((1 << 20, 8192, 0), ((1 << 28) + (1 << 20), 32, 1000)):
        p = rng.integers(1, 1 << 12, N).astype(np.uint64)   # filler far below the bin
        slots = rng.permutation(N)
        inside, above, low = slots[:M], slots[M:M + 1500], slots[M + 1500:M + 1500 + lower]
        p[inside] = base + rng.integers(0, width, M)
        p[above] = rng.integers(base + (1 << 24), 1 << 32, above.size)
        p[low] = (base & ~((1 << 21) - 1)) + rng.integers(0, 1000, lower)  # same first-pass bin, lower second-pass bin
        p = p.astype(np.uint32)
        t = gear.Table([1], capacity=N, T=T, residency=gear.GEAR_DEVICE, device=0)
        try:
            t.insert([np.zeros((N, T), np.uint8)], p)
            for K in (above.size + M, above.size + M - 1, above.size + M + 1, above.size + 1, above.size):
                say("TopK bin taken whole: base %#x, K=%d" % (base, K))
                idx, start, wt = t.select(gear.GEAR_TOPK, K, 1, 9, 0.0, weights=True)
                st, oidx, ostart, ow = oracle.select(oracle.TOPK, p, N, T, K, 1, 9, 0.0, True)
                np.testing.assert_array_equal(host(idx), oidx, err_msg="base %#x K=%d" % (base, K))
                np.testing.assert_array_equal(host(start), ostart)
                np.testing.assert_array_equal(host(wt), ow)
                assert t.sync() == (0 if st == oracle.OK else gear.GEAR_STATUS_NO_WEIGHT)
        finally:
            t.close()


@pytest.mark.parametrize("global_min", [False, True], ids=["batch-min", "global-min"])
def test_small_table_one_launch_and_tree_paths_alternate(global_min):
    """A table of at most 16384 slots selects in one launch for batches up
    to 2048 and through the sum tree above that; alternating the two with
    updates in between must give the oracle's draws and weights every time
    (the tree is rescanned when it went stale during one-launch selects)."""
    rng = np.random.default_rng(31)
    N, T = 16384, 3
    p = rng.integers(1, 1000, N).astype(np.uint32)
    p[rng.random(N) < 0.1] = 0
    t = gear.Table([2], capacity=N, T=T, residency=gear.GEAR_DEVICE, device=0)
    try:
        if global_min:
            t.set_options(gear.GEAR_OPT_IS_GLOBAL_MIN)
        t.insert([np.zeros((N, 2 * T), np.uint8)], p)
        for it, B in enumerate([100, 3000, 2048, 2049, 1, 4096, 777]):
            say("small table, B=%d, global_min=%s" % (B, global_min))
            seed = 1000 + it
            idx, start, wt = t.select(gear.GEAR_PRIORITIZED, B, 2, seed, 0.4, weights=True)
            st, oidx, ostart, ow = oracle.select(oracle.PRIORITIZED, p, N, T, B, 2, seed, 0.4, True,
                                                 global_min=global_min)
            assert st == oracle.OK
            np.testing.assert_array_equal(host(idx), oidx)
            np.testing.assert_array_equal(host(start), ostart)
            assert_weights(host(wt), ow)
            upd = rng.integers(0, N, 600).astype(np.int64)
            newp = rng.integers(0, 2000, 600).astype(np.uint32)
            t.update_priorities(torch.from_numpy(upd).to(cuda()), torch.from_numpy(newp).to(cuda()))
            oracle.update(p, upd, newp)
        np.testing.assert_array_equal(t.priorities(), p)
        assert t.sync() == 0
    finally:
        t.close()


# ---------------------------------------------------------------------------
# Seeded random configurations: table shapes, element sizes (all three
# element widths, narrow and wide windows), fills that wrap, strategies,
# batch sizes on both sides of the one-launch select's limit, window
# lengths and weights, each replayed against the oracle.
# ---------------------------------------------------------------------------

_KINDS = [(gen.BYTES, 1), (gen.DONE_U8, 1), (gen.INT_MOD, 4), (gen.NORMAL_F32, 4), (gen.UNIFORM_F32, 4),
          (gen.NORMAL_BF16, 2)]
_PRIOS = [U1000, BIG, gen.PrioDist(gen.PRIO_UNIFORM, 1, 3), gen.PrioDist(gen.PRIO_PARETO, 1.5, float(1 << 24)),
          gen.PrioDist(gen.PRIO_LOGNORMAL, 6.931471805599453, 1.0, float(1 << 24))]


def _random_workload(k):
    rng = np.random.default_rng(1000 + k)
    large = rng.random() < 0.35  # above the one-launch select's 16384 slots
    N = int(rng.integers(16385, 60001)) if large else int(np.exp(rng.uniform(0, np.log(16384))))
    T = int(rng.integers(1, 9 if large else 41))
    cols = []
    for c in range(int(rng.integers(0, 4))):
        kind, size = _KINDS[int(rng.integers(0, len(_KINDS)))]
        elems = int(rng.choice([1, 2, 3, 4, 8, 16, 17, 64, 96]))
        param = 16 if kind == gen.INT_MOD else 0
        cols.append(gen.Column("c%d" % c, kind, elems, param=param))
    # Keep the table within a few MB so the CPU oracle stays quick.
    while cols and N * T * sum(c.elem_bytes for c in cols) > (6 << 20):
        cols.pop()
    n_insert = int(rng.integers(1, 2 * N + 1))
    live = min(n_insert, N)
    strategies = tuple(int(s) for s in rng.permutation(5)[:int(rng.integers(1, 4))])
    B = int(rng.choice([1, 7, 256, 2048, 2049, 3000]))
    if any(s in (0, 1, 4) for s in strategies):
        B = min(B, live)
    L = int(rng.integers(1, T + 1))
    return _custom("random-%d" % k, N, T, cols, n_insert, _PRIOS[int(rng.integers(0, len(_PRIOS)))], B, L,
                   strategies=strategies, weights=bool(rng.integers(0, 2)), seed=int(rng.integers(1, 1 << 30)))


RANDOM = [_random_workload(k) for k in range(64)]
# The same kind of configurations with the table in pinned host memory,
# read zero-copy by the gather.
RANDOM += [dataclasses.replace(_random_workload(k), name="random-host-%d" % k, host_table=True)
           for k in range(64, 80)]


@pytest.mark.parametrize("w", RANDOM, ids=[w.name for w in RANDOM])
def test_random_configurations(w):
    _run_full(w, iterations=2)


RANDOM_OPT = [(_random_workload(k), gear.GEAR_OPT_INCREMENTAL_TREE) for k in range(80, 96)]
RANDOM_OPT += [(_random_workload(k), gear.GEAR_OPT_IS_GLOBAL_MIN) for k in range(96, 112)]
RANDOM_OPT += [(_random_workload(k), gear.GEAR_OPT_INCREMENTAL_TREE | gear.GEAR_OPT_IS_GLOBAL_MIN)
               for k in range(112, 120)]


@pytest.mark.parametrize("w,options", RANDOM_OPT, ids=["%s-opt%d" % (w.name, o) for w, o in RANDOM_OPT])
def test_random_configurations_with_options(w, options):
    _run_full(w, iterations=3, options=options)
