"""Checks of the synthetic-input generator (inputs only, not the method).

Philox4x32-10 is pinned by the known-answer vectors published with the
Random123 library (Salmon et al., SC 2011); the value recipes are checked
against torch/numpy conversions and loose distribution statistics.
"""
import numpy as np
import pytest
import torch

import gen
from gen import configs


def test_philox_known_answers():
    M = 0xFFFFFFFF
    assert gen.philox4x32_10([0, 0, 0, 0], [0, 0]) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert gen.philox4x32_10([M] * 4, [M, M]) == [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]
    assert gen.philox4x32_10([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344],
                             [0xA4093822, 0x299F31D0]) == [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]


def test_normal_recipe_moments_and_grid():
    col = gen.Column("x", gen.NORMAL_F32, 64)
    x = gen.fill_rows_cpu(col, 0, 1, 100, 0, 64).view(np.float32).astype(np.float64).ravel()
    assert abs(x.mean()) < 0.01 and abs(x.var() - 1.0) < 0.02
    assert np.all(np.abs(x) <= 6.0)
    assert np.all(x * 65536 == np.round(x * 65536))   # exact multiples of 2^-16


def test_bf16_matches_torch_round_to_nearest_even():
    f = gen.Column("x", gen.NORMAL_F32, 512)
    h = gen.Column("x", gen.NORMAL_BF16, 512)
    xf = gen.fill_rows_cpu(f, 3, 9, 20, 5, 4).view(np.float32)
    xh = gen.fill_rows_cpu(h, 3, 9, 20, 5, 4).view(np.uint16)
    ref = torch.from_numpy(xf.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(xh, ref)


def test_rtg_is_reverse_cumsum_of_reward():
    w = configs.DT
    T = 50
    rew = gen.fill_rows_cpu(w.columns[2], 2, w.seed, T, 10, 3).view(np.float32)
    rtg = gen.fill_rows_cpu(w.columns[3], 3, w.seed, T, 10, 3).view(np.float32)
    ref = np.cumsum(rew.astype(np.float64)[:, ::-1], axis=1)[:, ::-1].astype(np.float32)
    np.testing.assert_array_equal(rtg, ref)


def test_uniform_and_int_ranges():
    u = gen.fill_rows_cpu(gen.Column("a", gen.UNIFORM_F32, 6), 1, 2, 100, 0, 20).view(np.float32)
    assert u.min() >= -1.0 and u.max() < 1.0 and abs(u.mean()) < 0.02
    a = gen.fill_rows_cpu(gen.Column("a", gen.INT_MOD, 8, param=16), 1, 2, 100, 0, 20).view(np.int32)
    assert a.min() == 0 and a.max() == 15
    d = gen.fill_rows_cpu(gen.Column("d", gen.DONE_U8, 1), 4, 2, 30, 0, 5).reshape(5, 30)
    assert np.all(d[:, -1] == 1) and np.all(d[:, :-1] == 0)


def test_rows_are_pure_functions_of_insertion_number():
    col = gen.Column("o", gen.BYTES, 1000)
    a = gen.fill_rows_cpu(col, 0, 4, 7, 100, 10)
    b = gen.fill_rows_cpu(col, 0, 4, 7, 105, 2)
    np.testing.assert_array_equal(a[5:7], b)
    c = gen.fill_rows_cpu(col, 1, 4, 7, 105, 2)
    assert not np.array_equal(b, c)


@pytest.mark.parametrize("w", [configs.TINY, configs.SELECT_STRESS, configs.GATO_HOST, configs.MAT])
def test_priority_distributions(w):
    p = gen.insert_priorities(w.prio, w.seed, 0, 200000)
    assert p.min() >= 1
    if w.prio.kind == gen.PRIO_UNIFORM:
        assert p.max() <= w.prio.b and p.min() == w.prio.a
    elif w.prio.kind == gen.PRIO_PARETO:
        assert p.max() <= w.prio.b
        # P(p >= 2) = 2^-1.5 for floor(Pareto(1.5, x_m = 1))
        assert abs(np.mean(p >= 2) - 2 ** -1.5) < 0.01
    else:
        assert abs(np.median(p) - 1024) < 20
        assert p.max() <= w.prio.c
    q = gen.update_priorities(w.prio, w.seed, 0, 1000)
    assert not np.array_equal(q, p[:1000])
