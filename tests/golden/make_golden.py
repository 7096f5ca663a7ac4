"""Writes oracle_select_regression.txt: selection outputs of the oracle on
small fixed inputs, stored so that any later change to the oracle's
arithmetic shows up as a diff.  Calls only the oracle (inputs are literal).

Run:  python -m tests.golden.make_golden
"""
import os

import numpy as np

import oracle

CASES = [
    dict(name="prioritized_p10", strategy=oracle.PRIORITIZED,
         priority=[3, 0, 1, 4, 0, 0, 2, 5, 0, 1], next_seq=10, T=8, B=12, L=3, seed=2024, beta=0.4),
    dict(name="prioritized_big_weights", strategy=oracle.PRIORITIZED,
         priority=[0xFFFFFFFF, 1, 0, 0x80000000, 7], next_seq=5, T=1, B=8, L=1, seed=1, beta=1.0),
    dict(name="uniform_partial", strategy=oracle.UNIFORM,
         priority=[1] * 16, next_seq=11, T=30, B=10, L=30, seed=77, beta=0.0),
    dict(name="fifo_wrapped", strategy=oracle.FIFO,
         priority=[1] * 16, next_seq=37, T=5, B=16, L=2, seed=5, beta=0.0),
    dict(name="lifo_wrapped", strategy=oracle.LIFO,
         priority=[1] * 16, next_seq=37, T=5, B=7, L=5, seed=5, beta=0.0),
]


def run_case(c):
    p = np.array(c["priority"], dtype=np.uint32)
    st, idx, start, w = oracle.select(c["strategy"], p, c["next_seq"], c["T"], c["B"], c["L"],
                                      c["seed"], c["beta"], True)
    assert st == oracle.OK
    return [(int(i), int(s), float(x).hex()) for i, s, x in zip(idx, start, w)]


def main():
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_select_regression.txt")
    with open(path, "w") as f:
        f.write("# Oracle selection outputs on literal inputs (tests/golden/make_golden.py).\n")
        f.write("# format: case idx start weight(float hex)\n")
        for c in CASES:
            for i, s, x in run_case(c):
                f.write("%s %d %d %s\n" % (c["name"], i, s, x))


if __name__ == "__main__":
    main()
