"""Plain CPU oracle for experience-replay selection and collection.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the CPU-baseline leg of the benchmark may import this package.  The product
library never imports it and never falls back to it.

The arithmetic lives in ``oracle.c`` (plain single-threaded C, built with gcc
into ``liboracle.so``).  This module only marshals numpy arrays into it.
Each wrapper names the definition it follows; see ``oracle.c`` for the
passages of the GEAR paper (arXiv 2310.05205) each one restates.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

FIFO, LIFO, UNIFORM, PRIORITIZED, TOPK = 0, 1, 2, 3, 4
OK, INVAL, EMPTY, INSUFFICIENT, NO_WEIGHT = 0, -1, -3, -4, -6


def build(force=False):
    """Compile oracle.c with gcc (single-threaded, -O2, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
                               "-ffp-contract=off", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        u64, i64, i32, u32p = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        vp = ctypes.c_void_p
        L.oracle_mix64.argtypes = [u64]; L.oracle_mix64.restype = u64
        L.oracle_draw.argtypes = [u64, u64]; L.oracle_draw.restype = u64
        L.oracle_bounded.argtypes = [u64, u64]; L.oracle_bounded.restype = u64
        L.oracle_prefix_sum.argtypes = [vp, i64, vp]; L.oracle_prefix_sum.restype = u64
        L.oracle_upper_bound.argtypes = [vp, i64, u64]; L.oracle_upper_bound.restype = i64
        L.oracle_select.argtypes = [ctypes.c_int, vp, i64, u64, i32, i32, i32, u64, ctypes.c_float,
                                    vp, vp, vp, vp]
        L.oracle_select.restype = ctypes.c_int
        L.oracle_collect.argtypes = [i32, vp, vp, i64, i32, vp, vp, i32, i32, vp]
        L.oracle_collect.restype = ctypes.c_int
        L.oracle_update.argtypes = [vp, i64, vp, vp, i32]; L.oracle_update.restype = ctypes.c_int
        L.oracle_insert.argtypes = [i32, vp, vp, i64, i32, u64, i64, vp, vp, vp]
        L.oracle_insert.restype = u64
        L.oracle_translate.argtypes = [i64, i64, vp, vp]
        L.oracle_translate.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data if a is not None else None


def mix64(z):
    return lib().oracle_mix64(z)


def draw(seed, c):
    """Output number c of the splitmix64 stream seeded with `seed`."""
    return lib().oracle_draw(seed, c)


def bounded(u, n):
    """floor(u * n / 2^64)."""
    return lib().oracle_bounded(u, n)


def prefix_sum(p):
    """Inclusive prefix sum of uint32 priorities into uint64; returns (C, S)."""
    p = np.ascontiguousarray(p, dtype=np.uint32)
    C = np.empty(p.size, dtype=np.uint64)
    S = lib().oracle_prefix_sum(_ptr(p), p.size, _ptr(C))
    return C, S


def upper_bound(C, r):
    C = np.ascontiguousarray(C, dtype=np.uint64)
    return lib().oracle_upper_bound(_ptr(C), C.size, r)


def select(strategy, priority, next_seq, T, B, L, seed, beta=0.0, weights=False):
    """Returns (status, idx int64[B], start int32[B], w float32[B] or None)."""
    priority = np.ascontiguousarray(priority, dtype=np.uint32)
    N = priority.size
    idx = np.zeros(max(B, 0), dtype=np.int64)
    start = np.zeros(max(B, 0), dtype=np.int32)
    w = np.zeros(max(B, 0), dtype=np.float32) if weights else None
    C = np.empty(N, dtype=np.uint64) if strategy == PRIORITIZED else None
    st = lib().oracle_select(strategy, _ptr(priority), N, next_seq, T, B, L, seed,
                             ctypes.c_float(beta), _ptr(idx), _ptr(start), _ptr(w), _ptr(C))
    return st, idx, start, w


def collect(columns, T, idx, start, L):
    """columns: list of uint8 arrays shaped [N, T*E_c] (or [N, T, E_c]).
    Returns (status, list of uint8 arrays shaped [B, L*E_c])."""
    cols = [np.ascontiguousarray(c).reshape(c.shape[0], -1).view(np.uint8) for c in columns]
    N = cols[0].shape[0]
    E = np.array([c.shape[1] // T for c in cols], dtype=np.int64)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    start = np.ascontiguousarray(start, dtype=np.int32)
    B = idx.size
    outs = [np.zeros((B, L * int(e)), dtype=np.uint8) for e in E]
    bases = (ctypes.c_void_p * len(cols))(*[c.ctypes.data for c in cols])
    optrs = (ctypes.c_void_p * len(cols))(*[o.ctypes.data for o in outs])
    st = lib().oracle_collect(len(cols), bases, _ptr(E), N, T, _ptr(idx), _ptr(start), B, L, optrs)
    return st, outs


def update(priority, idx, newp):
    """In-place, batch order, last write wins.  Returns status."""
    assert priority.dtype == np.uint32 and priority.flags.c_contiguous
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    newp = np.ascontiguousarray(newp, dtype=np.uint32)
    return lib().oracle_update(_ptr(priority), priority.size, _ptr(idx), _ptr(newp), idx.size)


def translate(global_idx, capacity):
    """(shard, local) of a global index under equal-capacity sharding."""
    s = ctypes.c_int64(0)
    l = ctypes.c_int64(0)
    st = lib().oracle_translate(int(global_idx), int(capacity), ctypes.byref(s), ctypes.byref(l))
    if st != OK:
        raise ValueError("invalid index or capacity")
    return s.value, l.value


class Store:
    """Host-memory store driven through the oracle: columns [N, T*E_c] bytes,
    priorities uint32[N] and the insertion count."""

    def __init__(self, elem_bytes, N, T):
        self.E = [int(e) for e in elem_bytes]
        self.N, self.T = int(N), int(T)
        self.cols = [np.zeros((self.N, self.T * e), dtype=np.uint8) for e in self.E]
        self.priority = np.zeros(self.N, dtype=np.uint32)
        self.next_seq = 0

    def insert(self, rows, prio):
        """rows: list (per column) of uint8 arrays [n, T*E_c]; prio uint32[n]."""
        n = int(np.asarray(prio).size)
        rows = [np.ascontiguousarray(r).reshape(n, -1).view(np.uint8) for r in rows]
        prio = np.ascontiguousarray(prio, dtype=np.uint32)
        Ea = np.array(self.E, dtype=np.int64)
        bases = (ctypes.c_void_p * len(self.cols))(*[c.ctypes.data for c in self.cols])
        srcs = (ctypes.c_void_p * len(rows))(*[r.ctypes.data for r in rows])
        self.next_seq = lib().oracle_insert(len(self.cols), bases, _ptr(Ea), self.N, self.T,
                                            self.next_seq, n, srcs, _ptr(self.priority), _ptr(prio))

    def select(self, strategy, B, L, seed, beta=0.0, weights=False):
        return select(strategy, self.priority, self.next_seq, self.T, B, L, seed, beta, weights)

    def collect(self, idx, start, L, col_ids=None):
        cols = self.cols if col_ids is None else [self.cols[i] for i in col_ids]
        return collect(cols, self.T, idx, start, L)

    def update(self, idx, newp):
        return update(self.priority, idx, newp)
