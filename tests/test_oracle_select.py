"""Pins for the oracle's selection: prefix sum, search, the four strategies
and importance-sampling weights.

Weighted sampling is a prefix sum followed by a binary search for each
uniform number (GEAR Sec. 3.3, centralized selection); zero priority is never
selectable (Sec. 3.2, index manager).  The checks below compare the oracle
with numpy's cumsum/searchsorted, with brute-force enumeration of every
random number on tiny inputs, and with closed forms.
"""
import math

import numpy as np
import pytest

import oracle
from gen import STAMP, Column, fill_rows_cpu


def test_prefix_sum_matches_numpy_cumsum():
    rng = np.random.default_rng(0)
    for n in [1, 2, 255, 256, 257, 4096, 100003]:
        p = rng.integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32)
        C, S = oracle.prefix_sum(p)
        np.testing.assert_array_equal(C, np.cumsum(p, dtype=np.uint64))
        assert S == int(p.astype(np.uint64).sum())


def test_prefix_sum_does_not_wrap_at_32_bits():
    p = np.full(5000, 0xFFFFFFFF, dtype=np.uint32)
    C, S = oracle.prefix_sum(p)
    assert S == 5000 * 0xFFFFFFFF
    assert int(C[1]) == 2 * 0xFFFFFFFF


def test_upper_bound_matches_searchsorted_right():
    rng = np.random.default_rng(1)
    p = rng.integers(0, 20, size=3000).astype(np.uint32)
    p[100:400] = 0                        # a run of unselectable slots
    C, S = oracle.prefix_sum(p)
    probes = list(rng.integers(0, S, size=3000)) + [0, S - 1]
    probes += [int(c) for c in C[::37]] + [int(c) - 1 for c in C[::41] if c > 0]
    for r in probes:
        r = int(r)
        if r >= S:
            continue
        assert oracle.upper_bound(C, r) == int(np.searchsorted(C, r, side="right"))


def test_search_brute_force_every_random_number():
    # Over all r in [0, S) slot i is hit exactly p_i times; zero never.
    p = np.array([3, 0, 1, 4, 0, 0, 2, 5, 0, 1], dtype=np.uint32)
    C, S = oracle.prefix_sum(p)
    hits = np.zeros(p.size, dtype=np.int64)
    for r in range(S):
        hits[oracle.upper_bound(C, r)] += 1
    np.testing.assert_array_equal(hits, p.astype(np.int64))


def test_search_leading_and_trailing_zeros():
    p = np.array([0, 0, 0, 7, 0, 0], dtype=np.uint32)
    C, S = oracle.prefix_sum(p)
    assert {oracle.upper_bound(C, r) for r in range(S)} == {3}


def _draws_python(seed, B, S, span):
    """The draw definition evaluated with Python integers: r_b and start_b."""
    r = [(oracle.draw(seed, 2 * b) * S) >> 64 for b in range(B)]
    st = [(oracle.draw(seed, 2 * b + 1) * span) >> 64 for b in range(B)]
    return r, st


@pytest.mark.parametrize("N,B,seed", [(1, 5, 0), (300, 256, 7), (4096, 1000, 123456789)])
def test_prioritized_select_matches_library_construction(N, B, seed):
    rng = np.random.default_rng(N)
    p = rng.integers(1, 1000, size=N).astype(np.uint32)
    if N > 10:
        p[rng.integers(0, N, size=N // 5)] = 0
    T, L = 64, 20
    st, idx, start, w = oracle.select(oracle.PRIORITIZED, p, N, T, B, L, seed, 0.4, True)
    assert st == oracle.OK
    C = np.cumsum(p, dtype=np.uint64)
    S = int(C[-1])
    r, s = _draws_python(seed, B, S, T - L + 1)
    np.testing.assert_array_equal(idx, np.searchsorted(C, np.array(r, dtype=np.uint64), side="right"))
    np.testing.assert_array_equal(start, np.array(s, dtype=np.int32))
    assert np.all(p[idx] > 0)


def test_is_weights_closed_form():
    # (n*P(i))^-beta / max_b (n*P(b))^-beta  ==  (p_min / p_i)^beta
    rng = np.random.default_rng(9)
    N = 5000
    p = rng.integers(1, 1 << 24, size=N).astype(np.uint32)
    for beta in [0.0, 0.4, 1.0]:
        st, idx, start, w = oracle.select(oracle.PRIORITIZED, p, N, 1, 777, 1, 42, beta, True)
        assert st == oracle.OK
        pb = p[idx].astype(np.float64)
        closed = (pb.min() / pb) ** beta
        np.testing.assert_allclose(w.astype(np.float64), closed, rtol=1e-6, atol=0)
        assert np.all(w > 0) and np.all(w <= 1.0)
        assert w[np.argmin(pb)] == 1.0


def test_is_weights_global_minimum_closed_form():
    # Normalised by the largest weight of any selectable slot, i.e. at the
    # smallest non-zero priority of the whole table: (p_min_all / p_b)^beta.
    rng = np.random.default_rng(19)
    N = 3000
    p = rng.integers(50, 1 << 20, size=N).astype(np.uint32)
    p[rng.integers(0, N, size=300)] = 0
    p[1234] = 7                                     # the global minimum, rarely drawn
    for beta in [0.0, 0.4, 1.0]:
        st, idx, start, w = oracle.select(oracle.PRIORITIZED, p, N, 1, 500, 1, 8, beta, True, global_min=True)
        assert st == oracle.OK
        closed = (7.0 / p[idx].astype(np.float64)) ** beta
        np.testing.assert_allclose(w.astype(np.float64), closed, rtol=1e-6, atol=0)
        assert np.all(w <= 1.0)
    # When the batch holds the global minimum both normalisations agree.
    q = np.array([3, 3, 3, 3], dtype=np.uint32)
    a = oracle.select(oracle.PRIORITIZED, q, 4, 1, 64, 1, 2, 0.6, True)[3]
    b = oracle.select(oracle.PRIORITIZED, q, 4, 1, 64, 1, 2, 0.6, True, global_min=True)[3]
    np.testing.assert_array_equal(a, b)


def test_is_weights_use_live_count_and_total():
    # With one live trajectory per distinct priority the max weight belongs
    # to the smallest priority and n, S cancel: w = (p_min/p_b)^beta.
    p = np.array([5, 10, 20, 40], dtype=np.uint32)
    st, idx, start, w = oracle.select(oracle.PRIORITIZED, p, 4, 1, 4000, 1, 3, 0.5, True)
    assert st == oracle.OK
    for b in range(20):
        if p[idx[b]] == p[idx].min():
            assert w[b] == 1.0
        assert w[b] == pytest.approx(math.sqrt(p[idx].min() / p[idx[b]]), rel=1e-6)


def test_prioritized_chi_square_sanity():
    rng = np.random.default_rng(21)
    N = 64
    p = rng.integers(1, 100, size=N).astype(np.uint32)
    B = 1_000_000
    st, idx, _, _ = oracle.select(oracle.PRIORITIZED, p, N, 1, B, 1, 99, 0.0, False)
    assert st == oracle.OK
    obs = np.bincount(idx, minlength=N).astype(np.float64)
    exp = B * p.astype(np.float64) / p.sum()
    chi2 = float(((obs - exp) ** 2 / exp).sum())
    # 63 degrees of freedom: mean 63, sd ~11.2; 130 is ~6 sd out.
    assert chi2 < 130.0


def _stamped_store(N, T, n_insert):
    col = Column("stamp", STAMP, 1)
    store = oracle.Store([col.elem_bytes], N, T)
    rows = fill_rows_cpu(col, 0, 0, T, 0, n_insert)
    store.insert([rows], np.ones(n_insert, dtype=np.uint32))
    return store


def _stamp_k(store, idx):
    """Insertion numbers read back from the stamp column at step 0."""
    return store.cols[0].view(np.uint32).reshape(store.N, store.T, 2)[idx, 0, 0]


@pytest.mark.parametrize("n_insert", [5, 16, 37, 100])
def test_fifo_lifo_follow_insertion_order(n_insert):
    N, T = 16, 4
    store = _stamped_store(N, T, n_insert)
    live = min(n_insert, N)
    oldest = n_insert - live
    for B in [1, live // 2 or 1, live]:
        st, idx, start, _ = store.select(oracle.FIFO, B, 2, 5)
        assert st == oracle.OK
        np.testing.assert_array_equal(_stamp_k(store, idx), np.arange(oldest, oldest + B))
        st, idx, start, _ = store.select(oracle.LIFO, B, 2, 5)
        assert st == oracle.OK
        np.testing.assert_array_equal(_stamp_k(store, idx), np.arange(n_insert - 1, n_insert - 1 - B, -1))
        assert np.all((start >= 0) & (start <= T - 2))
    st, *_ = store.select(oracle.FIFO, live + 1, 2, 5)
    assert st == oracle.INSUFFICIENT
    st, *_ = store.select(oracle.LIFO, live + 1, 2, 5)
    assert st == oracle.INSUFFICIENT


def test_uniform_ranges_and_partial_fill():
    N, T, L = 1000, 50, 7
    store = _stamped_store(N, T, 300)          # 300 live of 1000
    st, idx, start, w = store.select(oracle.UNIFORM, 20000, L, 77, weights=True)
    assert st == oracle.OK
    assert idx.min() >= 0 and idx.max() < 300
    assert start.min() >= 0 and start.max() <= T - L
    assert len(np.unique(idx)) > 280 and len(np.unique(start)) == T - L + 1
    assert np.all(w == 1.0)
    st, idx, start, _ = store.select(oracle.UNIFORM, 100, T, 77)
    assert np.all(start == 0)


def _splitmix64_python(seed, c):
    """Output c of splitmix64 seeded with `seed`, in Python integers from the
    generator's published definition (state advanced by the golden gamma c+1
    times, then the two xor-shift-multiply rounds and a final xor-shift)."""
    m = (1 << 64) - 1
    z = (seed + (c + 1) * 0x9E3779B97F4A7C15) & m
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
    return z ^ (z >> 31)


def test_python_splitmix64_agrees_with_published_outputs():
    # Vigna's splitmix64.c from state 0; the same words as the oracle's pin.
    assert [_splitmix64_python(0, c) for c in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4,
                                                            0x06C45D188009454F]


@pytest.mark.parametrize("N,n_insert,seed", [(1000, 300, 77), (1000, 1000, 5), (64, 1000, 123456789),
                                             (1, 9, 3), (7, 7 + 3, (1 << 64) - 1)])
def test_uniform_index_draw_matches_definition(N, n_insert, seed):
    # Uniform over the n live slots: idx_b = floor(u_2b * n / 2^64), with u_c
    # output c of the stream (index draw on the even counter, window start on
    # the odd one).  Ring tables: partly filled (n < N) and wrapped (n = N).
    T, L, B = 12, 5, 2000
    store = _stamped_store(N, T, n_insert)
    n = min(n_insert, N)
    st, idx, start, w = store.select(oracle.UNIFORM, B, L, seed, weights=True)
    assert st == oracle.OK
    expect_idx = [(_splitmix64_python(seed, 2 * b) * n) >> 64 for b in range(B)]
    expect_start = [(_splitmix64_python(seed, 2 * b + 1) * (T - L + 1)) >> 64 for b in range(B)]
    np.testing.assert_array_equal(idx, np.array(expect_idx, dtype=np.int64))
    np.testing.assert_array_equal(start, np.array(expect_start, dtype=np.int32))
    assert np.all(w == 1.0)


@pytest.mark.parametrize("removal", [oracle.FIFO, oracle.LIFO])
def test_uniform_index_draw_on_a_commit_list(removal):
    # With an index manager the r-th draw picks the r-th oldest committed
    # index: idx_b = order[floor(u_2b * n / 2^64)], n the committed count.
    N, T, L, B, seed = 50, 6, 2, 1500, 4242
    m = oracle.IndexManager(N, removal, 40)
    prio = np.zeros(N, dtype=np.uint32)
    rng = np.random.default_rng(removal)
    committed = []                               # the commit order, kept by this test
    for step in range(12):
        st, got = m.allocate(int(rng.integers(1, 9)), prio)
        assert st == oracle.OK
        victims = [i for i in committed if prio[i] == 0]
        committed = [i for i in committed if i not in victims]
        order = list(rng.permutation(got))
        assert m.commit(order, np.full(len(order), 3, dtype=np.uint32), prio) == oracle.OK
        committed += [int(i) for i in order]
    np.testing.assert_array_equal(m.order(), committed)
    n = len(committed)
    st, idx, start, _ = oracle.select(oracle.UNIFORM, prio, 0, T, B, L, seed, order=m.order())
    assert st == oracle.OK
    expect = [committed[(_splitmix64_python(seed, 2 * b) * n) >> 64] for b in range(B)]
    np.testing.assert_array_equal(idx, np.array(expect, dtype=np.int64))


def test_window_start_matches_definition():
    p = np.ones(10, dtype=np.uint32)
    T, L, B, seed = 1000, 20, 300, 31337
    for strat in [oracle.FIFO, oracle.UNIFORM, oracle.PRIORITIZED]:
        st, idx, start, _ = oracle.select(strat, p, 10, T, min(B, 10) if strat == oracle.FIFO else B, L, seed)
        assert st == oracle.OK
        expect = [(oracle.draw(seed, 2 * b + 1) * (T - L + 1)) >> 64 for b in range(start.size)]
        np.testing.assert_array_equal(start, expect)


def test_select_errors():
    p = np.zeros(8, dtype=np.uint32)
    assert oracle.select(oracle.PRIORITIZED, p, 8, 4, 2, 1, 0)[0] == oracle.NO_WEIGHT
    p[3] = 1
    assert oracle.select(oracle.PRIORITIZED, p, 8, 4, 2, 5, 0)[0] == oracle.INVAL      # L > T
    assert oracle.select(oracle.PRIORITIZED, p, 8, 4, 0, 1, 0)[0] == oracle.INVAL      # B = 0
    assert oracle.select(oracle.UNIFORM, p, 0, 4, 2, 1, 0)[0] == oracle.EMPTY          # nothing inserted
    assert oracle.select(9, p, 8, 4, 2, 1, 0)[0] == oracle.INVAL
    st, idx, _, _ = oracle.select(oracle.PRIORITIZED, p, 8, 4, 50, 1, 0)
    assert st == oracle.OK and np.all(idx == 3)


def _topk_numpy(p, K):
    """TopK by numpy's lexsort: priority descending, then slot ascending,
    among slots with non-zero priority."""
    cand = np.nonzero(p)[0]
    order = np.lexsort((cand, -p[cand].astype(np.int64)))
    sel = cand[order][:K]
    return np.concatenate([sel, -np.ones(K - sel.size, dtype=np.int64)])


@pytest.mark.parametrize("N,K,hi", [(1, 1, 5), (300, 64, 3), (5000, 777, 1000), (4096, 4096, 2), (100000, 8192, 1 << 32)])
def test_topk_matches_lexsort(N, K, hi):
    rng = np.random.default_rng(N + K)
    p = rng.integers(0, hi, size=N, dtype=np.uint64).astype(np.uint32)   # zeros and many ties
    T, L = 10, 3
    st, idx, start, w = oracle.select(oracle.TOPK, p, N, T, K, L, 12345, 0.0, True)
    ref = _topk_numpy(p, K)
    np.testing.assert_array_equal(idx, ref)
    assert st == (oracle.OK if np.count_nonzero(p) >= K else oracle.NO_WEIGHT)
    valid = idx >= 0
    assert np.all(w[valid] == 1.0) and np.all(w[~valid] == 0.0)
    expect = [(oracle.draw(12345, 2 * b + 1) * (T - L + 1)) >> 64 for b in range(K)]
    np.testing.assert_array_equal(start[valid], np.array(expect)[valid])
    assert np.all(start[~valid] == 0)


def test_topk_brute_force_small():
    # Every permutation-free check: the selected set is the K largest, ordered,
    # and no unselected slot beats a selected one.
    p = np.array([4, 0, 4, 1, 9, 4, 0, 2, 9, 1], dtype=np.uint32)
    st, idx, _, _ = oracle.select(oracle.TOPK, p, p.size, 1, 6, 1, 0)
    assert st == oracle.OK
    assert list(idx) == [4, 8, 0, 2, 5, 7]
    st, idx, _, _ = oracle.select(oracle.TOPK, p, p.size, 1, 9, 1, 0)
    assert st == oracle.NO_WEIGHT and list(idx) == [4, 8, 0, 2, 5, 7, 3, 9, -1]
