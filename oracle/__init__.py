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


class _Im(ctypes.Structure):
    """Mirror of the oracle's index-manager struct (orc_im)."""
    _fields_ = [("N", ctypes.c_int64), ("removal", ctypes.c_int), ("max_sel", ctypes.c_int64),
                ("free_q", ctypes.POINTER(ctypes.c_int64)), ("n_free", ctypes.c_int64),
                ("committed", ctypes.POINTER(ctypes.c_int64)), ("n_committed", ctypes.c_int64),
                ("n_pending", ctypes.c_int64), ("state", ctypes.POINTER(ctypes.c_uint8))]


IM_FREE, IM_PENDING, IM_COMMITTED = 0, 1, 2
_NO_ORDER = np.zeros(1, dtype=np.int64)

_lib = None


def lib():
    global _lib
    if _lib is None:
        # ORACLE_LIB names another build of oracle.c to load instead; the
        # mutation test loads deliberately broken builds through it.
        path = os.environ.get("ORACLE_LIB") or build()
        L = ctypes.CDLL(path)
        u64, i64, i32, u32p = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        vp = ctypes.c_void_p
        L.oracle_mix64.argtypes = [u64]; L.oracle_mix64.restype = u64
        L.oracle_draw.argtypes = [u64, u64]; L.oracle_draw.restype = u64
        L.oracle_bounded.argtypes = [u64, u64]; L.oracle_bounded.restype = u64
        L.oracle_prefix_sum.argtypes = [vp, i64, vp]; L.oracle_prefix_sum.restype = u64
        L.oracle_upper_bound.argtypes = [vp, i64, u64]; L.oracle_upper_bound.restype = i64
        L.oracle_select.argtypes = [ctypes.c_int, vp, i64, u64, vp, i64, i32, i32, i32, u64, ctypes.c_float,
                                    ctypes.c_int, vp, vp, vp, vp]
        L.oracle_select.restype = ctypes.c_int
        L.oracle_collect.argtypes = [i32, vp, vp, i64, i32, vp, vp, i32, i32, vp]
        L.oracle_collect.restype = ctypes.c_int
        L.oracle_update.argtypes = [vp, i64, vp, vp, i32]; L.oracle_update.restype = ctypes.c_int
        L.oracle_insert.argtypes = [i32, vp, vp, i64, i32, u64, i64, vp, vp, vp]
        L.oracle_insert.restype = u64
        L.oracle_translate.argtypes = [i64, i64, vp, vp]
        L.oracle_translate.restype = ctypes.c_int
        imp = ctypes.POINTER(_Im)
        L.oracle_im_init.argtypes = [imp, i64, ctypes.c_int, i64]; L.oracle_im_init.restype = ctypes.c_int
        L.oracle_im_free.argtypes = [imp]; L.oracle_im_free.restype = None
        L.oracle_im_allocate.argtypes = [imp, i64, vp, vp]; L.oracle_im_allocate.restype = ctypes.c_int
        L.oracle_im_commit.argtypes = [imp, i64, vp, vp, vp]; L.oracle_im_commit.restype = ctypes.c_int
        L.oracle_im_update.argtypes = [imp, vp, vp, vp, i32]; L.oracle_im_update.restype = ctypes.c_int
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


def select(strategy, priority, next_seq, T, B, L, seed, beta=0.0, weights=False, order=None, global_min=False):
    """Returns (status, idx int64[B], start int32[B], w float32[B] or None).
    `order`: the committed slots of an index manager, oldest first (FIFO,
    LIFO and uniform pick from it); None for the ring state `next_seq`.
    `global_min`: IS weights normalised over every non-zero priority instead
    of the batch."""
    priority = np.ascontiguousarray(priority, dtype=np.uint32)
    N = priority.size
    idx = np.zeros(max(B, 0), dtype=np.int64)
    start = np.zeros(max(B, 0), dtype=np.int32)
    w = np.zeros(max(B, 0), dtype=np.float32) if weights else None
    C = np.empty(N, dtype=np.uint64) if strategy == PRIORITIZED else None
    if order is not None:
        order = np.ascontiguousarray(order, dtype=np.int64)
        # A non-NULL pointer even for an empty list (never read then).
        optr, nord = (_ptr(order) if order.size else _ptr(_NO_ORDER)), order.size
    else:
        optr, nord = None, 0
    st = lib().oracle_select(strategy, _ptr(priority), N, next_seq, optr, nord, T, B, L, seed,
                             ctypes.c_float(beta), 1 if global_min else 0, _ptr(idx), _ptr(start), _ptr(w), _ptr(C))
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


class IndexManager:
    """The oracle's index manager: a free-index queue, a per-index state and
    the committed indices in commit order, with FIFO or LIFO removal and a
    maximum of selectable indices (oracle_im_* in oracle.c)."""

    def __init__(self, N, removal, max_sel):
        self._m = _Im()
        st = lib().oracle_im_init(ctypes.byref(self._m), int(N), int(removal), int(max_sel))
        if st != OK:
            raise ValueError("invalid index-manager parameters")

    def __del__(self):
        if getattr(self, "_m", None) is not None and lib is not None:
            lib().oracle_im_free(ctypes.byref(self._m))
            self._m = None

    @property
    def n_committed(self):
        return self._m.n_committed

    @property
    def n_pending(self):
        return self._m.n_pending

    @property
    def n_free(self):
        return self._m.n_free

    def order(self):
        """Committed indices, oldest commit first (a copy)."""
        return np.ctypeslib.as_array(self._m.committed, shape=(self._m.N,))[:self._m.n_committed].copy()

    def free_queue(self):
        return np.ctypeslib.as_array(self._m.free_q, shape=(self._m.N,))[:self._m.n_free].copy()

    def state(self):
        return np.ctypeslib.as_array(self._m.state, shape=(self._m.N,)).copy()

    def allocate(self, n, priority):
        """Returns (status, idx int64[n]); victims' priorities are zeroed."""
        assert priority.dtype == np.uint32 and priority.flags.c_contiguous
        idx = np.zeros(max(int(n), 1), dtype=np.int64)
        st = lib().oracle_im_allocate(ctypes.byref(self._m), int(n), _ptr(idx), _ptr(priority))
        return st, idx[:int(n)]

    def commit(self, idx, prio, priority):
        assert priority.dtype == np.uint32 and priority.flags.c_contiguous
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        prio = np.ascontiguousarray(prio, dtype=np.uint32)
        return lib().oracle_im_commit(ctypes.byref(self._m), idx.size, _ptr(idx), _ptr(prio), _ptr(priority))

    def update(self, priority, idx, newp):
        assert priority.dtype == np.uint32 and priority.flags.c_contiguous
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        newp = np.ascontiguousarray(newp, dtype=np.uint32)
        return lib().oracle_im_update(ctypes.byref(self._m), _ptr(priority), _ptr(idx), _ptr(newp), idx.size)


class Store:
    """Host-memory store driven through the oracle: columns [N, T*E_c] bytes,
    priorities uint32[N] and the insertion count; optionally managed by an
    IndexManager (use_allocator) instead of the ring."""

    def __init__(self, elem_bytes, N, T):
        self.E = [int(e) for e in elem_bytes]
        self.N, self.T = int(N), int(T)
        self.cols = [np.zeros((self.N, self.T * e), dtype=np.uint8) for e in self.E]
        self.priority = np.zeros(self.N, dtype=np.uint32)
        self.next_seq = 0
        self.im = None

    def use_allocator(self, removal, max_sel):
        assert self.next_seq == 0 and self.im is None
        self.im = IndexManager(self.N, removal, max_sel)

    def allocate(self, n):
        return self.im.allocate(n, self.priority)

    def write(self, idx, rows):
        """Writes rows[c][r] into block idx[r] of column c (in place)."""
        for c, r in enumerate(rows):
            self.cols[c][np.asarray(idx, dtype=np.int64)] = np.ascontiguousarray(r).reshape(len(idx), -1).view(np.uint8)

    def commit(self, idx, prio):
        return self.im.commit(idx, prio, self.priority)

    def insert(self, rows, prio):
        """rows: list (per column) of uint8 arrays [n, T*E_c]; prio uint32[n].
        With an index manager: one allocate of n, the writes, one commit."""
        n = int(np.asarray(prio).size)
        rows = [np.ascontiguousarray(r).reshape(n, -1).view(np.uint8) for r in rows]
        prio = np.ascontiguousarray(prio, dtype=np.uint32)
        if self.im is not None:
            st, idx = self.allocate(n)
            if st != OK:
                return st
            self.write(idx, rows)
            st = self.commit(idx, prio)
            self.next_seq += n
            return st
        Ea = np.array(self.E, dtype=np.int64)
        bases = (ctypes.c_void_p * len(self.cols))(*[c.ctypes.data for c in self.cols])
        srcs = (ctypes.c_void_p * len(rows))(*[r.ctypes.data for r in rows])
        self.next_seq = lib().oracle_insert(len(self.cols), bases, _ptr(Ea), self.N, self.T,
                                            self.next_seq, n, srcs, _ptr(self.priority), _ptr(prio))

    def select(self, strategy, B, L, seed, beta=0.0, weights=False, global_min=False):
        order = self.im.order() if self.im is not None else None
        return select(strategy, self.priority, self.next_seq, self.T, B, L, seed, beta, weights, order, global_min)

    def collect(self, idx, start, L, col_ids=None):
        cols = self.cols if col_ids is None else [self.cols[i] for i in col_ids]
        return collect(cols, self.T, idx, start, L)

    def update(self, idx, newp):
        if self.im is not None:
            return self.im.update(self.priority, idx, newp)
        return update(self.priority, idx, newp)
