"""Synthetic workloads shaped like the paper's experiments.

Each workload is a table (columns, capacity N, steps T), an insertion count,
a priority distribution and a selection request.  The real datasets behind
the paper's experiments (D4RL hopper for the decision-transformer shape,
Gato's offline data, StarCraft II multi-agent trajectories; Sec. 4.3) are not
used: these seeded tables stand in for them with the same shapes and value
distributions.
"""
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

from . import (BYTES, DONE_U8, INT_MOD, NORMAL_BF16, NORMAL_F32, PRIO_LOGNORMAL, PRIO_PARETO,
               PRIO_UNIFORM, RTG_F32, STAMP, UNIFORM_F32, Column, PrioDist)

FIFO, LIFO, UNIFORM, PRIORITIZED, TOPK = 0, 1, 2, 3, 4


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    N: int
    T: int
    columns: Tuple[Column, ...]
    n_insert: int
    prio: PrioDist
    strategies: Tuple[int, ...]
    B: int
    L: int
    beta: float = 0.4
    weights: bool = False
    iterations: int = 1
    host_table: bool = False

    @property
    def elem_bytes(self):
        return [c.elem_bytes for c in self.columns]

    @property
    def window_bytes(self):
        return sum(self.L * e for e in self.elem_bytes)

    @property
    def table_bytes(self):
        return self.N * self.T * sum(self.elem_bytes)


# Tiny prioritized replay: N=4096 x T=64, full 64-step trajectories.
TINY = Workload(
    name="tiny-prioritized N=4096 T=64 B=256 L=64",
    seed=1, N=4096, T=64,
    columns=(Column("obs", NORMAL_F32, 64, dtype="f32"),
             Column("action", INT_MOD, 1, param=1 << 31, dtype="i32"),
             Column("reward", NORMAL_F32, 1, dtype="f32"),
             Column("done", DONE_U8, 1, dtype="u8")),
    n_insert=4096, prio=PrioDist(PRIO_UNIFORM, 1, 1000),
    strategies=(PRIORITIZED,), B=256, L=64, weights=True)

# Decision-transformer shape, HBM table, ring wrapped by N/8 insertions.
DT = Workload(
    name="dt-windows N=65536 T=1000 B=512 L=20",
    seed=2, N=65536, T=1000,
    columns=(Column("obs", NORMAL_F32, 17, dtype="f32"),
             Column("action", UNIFORM_F32, 6, dtype="f32"),
             Column("reward", NORMAL_F32, 1, dtype="f32"),
             Column("rtg", RTG_F32, 1, param=2, dtype="f32")),
    n_insert=65536 + 65536 // 8, prio=PrioDist(PRIO_UNIFORM, 1, 1000),
    strategies=(UNIFORM, FIFO, LIFO), B=512, L=20)

# The same table, whole trajectories (L = T): 51.2 MB gathered per batch.
DT_FULL = Workload(
    name="dt-full-trajectories N=65536 T=1000 B=512 L=1000",
    seed=2, N=65536, T=1000, columns=DT.columns, n_insert=DT.n_insert, prio=DT.prio,
    strategies=(UNIFORM, FIFO, LIFO), B=512, L=1000)

# Selection-only stress: 2^22 Pareto(1.5) priorities, 100 iterations.
SELECT_STRESS = Workload(
    name="selection-stress N=4194304 B=8192 x100",
    seed=3, N=1 << 22, T=1, columns=(),
    n_insert=1 << 22, prio=PrioDist(PRIO_PARETO, 1.5, float(1 << 24)),
    strategies=(PRIORITIZED,), B=8192, L=1, weights=True, iterations=100)

# Gato-like image trajectories in pinned host memory, read zero-copy.
GATO_HOST = Workload(
    name="gato-host-zero-copy N=20000 T=128 B=1024 L=64",
    seed=4, N=20000, T=128,
    columns=(Column("obs", BYTES, 64 * 64 * 3, dtype="u8"),
             Column("action", INT_MOD, 1, param=18, dtype="i32"),
             Column("reward", NORMAL_F32, 1, dtype="f32")),
    n_insert=20000, prio=PrioDist(PRIO_UNIFORM, 1, 1 << 16),
    strategies=(PRIORITIZED,), B=1024, L=64, weights=True, host_table=True)

# MAT-shaped end-to-end iteration, HBM table: 8 agents x bf16[64] obs.
MAT = Workload(
    name="mat-end-to-end N=500000 T=200 B=8192 L=32",
    seed=5, N=500000, T=200,
    columns=(Column("obs", NORMAL_BF16, 8 * 64, dtype="bf16"),
             Column("action", INT_MOD, 8, param=16, dtype="i32"),
             Column("reward", NORMAL_F32, 1, dtype="f32")),
    n_insert=500000, prio=PrioDist(PRIO_LOGNORMAL, 6.931471805599453, 1.0, float(1 << 24)),
    strategies=(PRIORITIZED,), B=8192, L=32, weights=True, iterations=20)

# TopK over the selection-stress priorities: the 8192 highest of 2^22.
TOPK_STRESS = Workload(
    name="topk-stress N=4194304 K=8192",
    seed=3, N=1 << 22, T=1, columns=(),
    n_insert=1 << 22, prio=PrioDist(PRIO_PARETO, 1.5, float(1 << 24)),
    strategies=(TOPK,), B=8192, L=1, weights=False, iterations=100)

ALL = (TINY, DT, DT_FULL, SELECT_STRESS, GATO_HOST, MAT, TOPK_STRESS)
