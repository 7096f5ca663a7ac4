"""Shared helpers of the GPU parity tests: building the HIP-side table and
the oracle-side expectations from the same generated inputs."""
import sys

import numpy as np
import torch

import gen
import oracle
from gen.fill import fill_table
from paper_2310_05205_amd import gear

DEV = 0


def say(msg):
    """Progress line naming the case before a GPU step."""
    print(msg, file=sys.stderr, flush=True)


def cuda():
    return torch.device("cuda", DEV)


def host(t):
    return t.detach().cpu().numpy()


def gpu_table(w, residency=None, options=0):
    """HIP-side table holding all of w's insertions."""
    if residency is None:
        residency = gear.GEAR_HOST_PINNED if w.host_table else gear.GEAR_DEVICE
    t = gear.Table(w.elem_bytes, w.N, w.T, residency, DEV)
    if options:
        t.set_options(options)
    fill_table(w, lambda n, ptrs, prio: t.insert(ptrs, prio), device=DEV)
    return t


def oracle_priorities(w):
    """Priority array after all of w's insertions, via the oracle's ring."""
    s = oracle.Store([], w.N, w.T)
    s.insert([], gen.insert_priorities(w.prio, w.seed, 0, w.n_insert))
    return s.priority.copy(), s.next_seq


def oracle_store(w):
    """Full oracle store (small workloads only)."""
    s = oracle.Store(w.elem_bytes, w.N, w.T)
    rows = [gen.fill_rows_cpu(c, ci, w.seed, w.T, 0, w.n_insert) for ci, c in enumerate(w.columns)]
    s.insert(rows, gen.insert_priorities(w.prio, w.seed, 0, w.n_insert))
    return s


def oracle_windows(w, idx, start, L, next_seq, sample, col_ids=None):
    """Oracle collection of the sampled draws from a compact table holding
    only the trajectories those draws select (regenerated on the CPU)."""
    cols = list(range(len(w.columns))) if col_ids is None else list(col_ids)
    ks = gen.slot_insertion(np.asarray(idx)[sample], next_seq, w.N)
    rows = [gen.fill_rows_list_cpu(w.columns[c], c, w.seed, w.T, ks) for c in cols]
    st, outs = oracle.collect(rows, w.T, np.arange(len(sample)), np.asarray(start)[sample], L)
    assert st == oracle.OK
    return outs


def assert_weights(gpu_w, orc_w):
    np.testing.assert_allclose(gpu_w.astype(np.float64), orc_w.astype(np.float64), rtol=1e-6, atol=0)
