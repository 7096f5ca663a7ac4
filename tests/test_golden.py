"""Golden fixtures: the paper's printed worked example and the oracle's
stored regression values (written by tests/golden/make_golden.py, which
calls only the oracle)."""
import os

import numpy as np

import oracle

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rows(name):
    with open(os.path.join(GOLD, name)) as f:
        return [l.split() for l in f if l.strip() and not l.startswith("#")]


def test_paper_collection_example_index_translation():
    rows = [tuple(int(x) for x in r) for r in _rows("collect_example_index_translation.txt")]
    for g, shard, local in rows:
        assert oracle.translate(g, 24) == (shard, local)
    # 24 is the only capacity that reproduces the printed lists.
    fits = [cap for cap in range(1, 100)
            if all(oracle.translate(g, cap) == (s, l) for g, s, l in rows)]
    assert fits == [24]


def test_oracle_regression_fixture():
    from tests.golden.make_golden import CASES, run_case
    stored = {}
    for r in _rows("oracle_select_regression.txt"):
        stored.setdefault(r[0], []).append(r[1:])
    assert set(stored) == {c["name"] for c in CASES}
    for case in CASES:
        got = run_case(case)
        assert [list(map(str, g)) for g in got] == stored[case["name"]], case["name"]
