"""The oracle's pins catch plausible mistakes in the oracle itself.

Each case plants one mistake in a copy of oracle/oracle.c (a dropped term, an
off-by-one, a reversed order, a wrong bound, a swapped strategy ...), builds
that copy with gcc into a temporary directory, and runs the oracle's
independent pins against it in a child process (ORACLE_LIB points the oracle
package at the broken build).  Every planted mistake must fail at least one
pin.  The pins run here are the ones fixed by the paper and by mathematics:
splitmix64 and multiply-high properties, closed forms, brute force on tiny
inputs, library routines, invariants and the paper's worked collection
example.  The stored regression fixture is left out: it was written by the
oracle and would catch any change trivially.

The source file itself is never modified, and nothing here runs on a GPU.
"""
import concurrent.futures
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
PINS = ["tests/test_oracle_rng.py", "tests/test_oracle_select.py", "tests/test_oracle_collect_update.py",
        "tests/test_oracle_allocator.py",
        "tests/test_golden.py::test_paper_collection_example_index_translation"]
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math", "-ffp-contract=off"]

# (name, text in oracle.c, text that replaces it).  Each text occurs once.
MUTATIONS = [
    # counter-based draws
    ("mix64 first shift", "z = (z ^ (z >> 30)) *", "z = (z ^ (z >> 29)) *"),
    ("draw counter off by one", "seed + (c + 1u) * 0x9E37", "seed + c * 0x9E37"),
    ("bounded keeps a low bit", "(uint64_t)(prod >> 64)", "(uint64_t)(prod >> 63)"),
    # prefix sum and search
    ("prefix sum in 32 bits", "acc += (uint64_t)p[i];", "acc = (uint32_t)(acc + p[i]);"),
    ("exclusive prefix", "        acc += (uint64_t)p[i];\n        C[i] = acc;",
     "        C[i] = acc;\n        acc += (uint64_t)p[i];"),
    ("lower bound instead of upper bound", "if (C[mid] > r)", "if (C[mid] >= r)"),
    ("no-weight check dropped", "if (S == 0)\n            return ORC_NO_WEIGHT;", ""),
    # FIFO / LIFO / uniform
    ("FIFO skips the oldest", "k = next_seq - (uint64_t)n + (uint64_t)b;",
     "k = next_seq - (uint64_t)n + (uint64_t)b + 1u;"),
    ("LIFO starts past the newest", "k = next_seq - 1u - (uint64_t)b;", "k = next_seq - (uint64_t)b;"),
    ("FIFO/LIFO bound on capacity", "if ((int64_t)B > n)\n            return ORC_INSUFFICIENT;",
     "if ((int64_t)B > N)\n            return ORC_INSUFFICIENT;"),
    ("LIFO over the commit list in FIFO order", "order[n - 1 - b]", "order[b]"),
    ("uniform over capacity", "oracle_draw(seed, 2u * (uint64_t)b), (uint64_t)n);",
     "oracle_draw(seed, 2u * (uint64_t)b), (uint64_t)N);"),
    ("uniform index on the start's counter", "oracle_draw(seed, 2u * (uint64_t)b), (uint64_t)n);",
     "oracle_draw(seed, 2u * (uint64_t)b + 1u), (uint64_t)n);"),
    ("uniform index on counter b", "oracle_draw(seed, 2u * (uint64_t)b), (uint64_t)n);",
     "oracle_draw(seed, (uint64_t)b), (uint64_t)n);"),
    ("uniform ignores the commit list", "idx[b] = order != NULL ? order[r] : r;", "idx[b] = r;"),
    # window starts
    ("start reuses the index draw", "start[b] = (int32_t)oracle_bounded(oracle_draw(seed, 2u * (uint64_t)b + 1u),\n"
     "                                           (uint64_t)(T - L + 1));",
     "start[b] = (int32_t)oracle_bounded(oracle_draw(seed, 2u * (uint64_t)b),\n"
     "                                           (uint64_t)(T - L + 1));"),
    ("start range one short", "                                           (uint64_t)(T - L + 1));",
     "                                           (uint64_t)(T - L));"),
    # IS weights
    ("weight exponent sign", "double v = pow(x, -(double)beta);\n                w[b] = (float)(v / wmax);",
     "double v = pow(x, (double)beta);\n                w[b] = (float)(v / wmax);"),
    ("weights not normalised", "w[b] = (float)(v / wmax);", "w[b] = (float)(v);"),
    ("global normalisation ignored", "if (global_min) {", "if (0) {"),
    # TopK
    ("TopK ascending", "return x->p > y->p ? -1 : 1;", "return x->p < y->p ? -1 : 1;"),
    ("TopK tie-break on the higher slot", "return x->i < y->i ? -1 : (x->i > y->i ? 1 : 0);",
     "return x->i > y->i ? -1 : (x->i < y->i ? 1 : 0);"),
    ("TopK takes zero priorities", "            if (priority[i] > 0) {\n                cand[ncand].p",
     "            if (priority[i] >= 0) {\n                cand[ncand].p"),
    # collection
    ("window ignores its start", "((idx[b] * (int64_t)T) + start[b] + t) * E", "((idx[b] * (int64_t)T) + t) * E"),
    ("output step-major", "uint8_t *dst = out[c] + (((int64_t)b * L) + t) * E;",
     "uint8_t *dst = out[c] + (((int64_t)t * B) + b) * E;"),
    ("missing window rejected", "if (idx[b] != -1 && (idx[b] < 0", "if ((idx[b] < 0"),
    # update and insertion
    ("update applied in reverse", "for (b = 0; b < B; b++)\n        priority[idx[b]] = newp[b];",
     "for (b = B - 1; b >= 0; b--)\n        priority[idx[b]] = newp[b];"),
    ("update bound off by one", "    for (b = 0; b < B; b++)\n        if (idx[b] < 0 || idx[b] >= N)\n            return ORC_INVAL;\n"
     "    for (b = 0; b < B; b++)\n        priority",
     "    for (b = 0; b < B; b++)\n        if (idx[b] < 0 || idx[b] > N)\n            return ORC_INVAL;\n"
     "    for (b = 0; b < B; b++)\n        priority"),
    ("insert ignores the ring position", "uint64_t slot = (next_seq + (uint64_t)r) % (uint64_t)N;",
     "uint64_t slot = ((uint64_t)r) % (uint64_t)N;"),
    ("insert reads the slot's row", "src[c] + r * block", "src[c] + (int64_t)slot * block"),
    # index manager
    ("removal strategies swapped", "if (m->removal == ORC_FIFO) {", "if (m->removal != ORC_FIFO) {"),
    ("pending indices not counted", "m->n_committed + m->n_pending >= m->max_sel)",
     "m->n_committed >= m->max_sel)"),
    ("released victim keeps its priority", "    priority[v] = 0;\n", ""),
    ("late update of a released index", "if (m->state[idx[b]] == ORC_IM_COMMITTED)", "if (1)"),
    ("commit accepts a repeated index", "            if (idx[q] == idx[r])\n                return ORC_INVAL;",
     "            (void)q;"),
    # index translation
    ("shard and local swapped", "*shard = global / capacity;\n    *local = global % capacity;",
     "*shard = global % capacity;\n    *local = global / capacity;"),
]


def _build(source, path):
    src = path + ".c"
    with open(src, "w") as f:
        f.write(source)
    subprocess.run(["gcc"] + CFLAGS + ["-o", path, src, "-lm"], check=True, capture_output=True)


def _run_pins(lib_path):
    env = dict(os.environ, ORACLE_LIB=lib_path, PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider"] + PINS,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    return r.returncode, r.stdout[-2000:]


def test_every_planted_mistake_fails_a_pin(tmp_path):
    with open(SRC) as f:
        original = f.read()
    for name, old, _ in MUTATIONS:
        assert original.count(old) == 1, "mutation %r no longer matches oracle.c exactly once" % name

    # The unchanged oracle, built the same way, passes every pin.
    base = str(tmp_path / "liboracle_base.so")
    _build(original, base)
    rc, out = _run_pins(base)
    assert rc == 0, "the pins fail on the unchanged oracle:\n" + out

    def one(k):
        name, old, new = MUTATIONS[k]
        path = str(tmp_path / ("liboracle_m%02d.so" % k))
        _build(original.replace(old, new), path)
        rc, out = _run_pins(path)
        return name, rc, out

    workers = max(1, min(4, (os.cpu_count() or 1) // 2))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(one, range(len(MUTATIONS))))
    survivors = [name for name, rc, _ in results if rc == 0]
    assert not survivors, "planted mistakes that no pin caught: %s" % survivors
    # A failed pin exits with 1; a mistake that makes the oracle crash ends
    # the child with a signal.  A usage or collection error (2 to 5) would
    # not be a pin failing.
    bad = [(n, rc, out[-300:]) for n, rc, out in results if not (rc == 1 or rc < 0)]
    assert not bad, bad
