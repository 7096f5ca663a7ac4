"""Seeded synthetic inputs shared by the library's tests, the oracle and the
benchmark.

This package produces inputs only (column contents, initial priorities and
the new priorities given to updates); it contains none of the replay method's
arithmetic.  ``gen.c`` is the CPU implementation (gcc, OpenMP over rows) and
``gen_gpu.hip`` the byte-identical GPU implementation used to fill large
tables.  The definitions of every value are at the top of ``gen.c``.
"""
import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_CPU_SRC = os.path.join(_HERE, "gen.c")
_CPU_LIB = os.path.join(_HERE, "libgen_cpu.so")
_GPU_SRC = os.path.join(_HERE, "gen_gpu.hip")
_GPU_LIB = os.path.join(_HERE, "libgen_gpu.so")

BYTES, NORMAL_F32, UNIFORM_F32, INT_MOD, NORMAL_BF16, DONE_U8, RTG_F32, STAMP = range(8)
PRIO_UNIFORM, PRIO_PARETO, PRIO_LOGNORMAL = range(3)
PRIO_STREAM = 0xFFFF          # stream id of the initial priority of insertion k
UPDATE_STREAM0 = 0x10000      # stream id 0x10000 + t: new priorities of iteration t

_ESZ = {BYTES: 1, DONE_U8: 1, NORMAL_BF16: 2, STAMP: 8}


def elem_size(kind):
    return _ESZ.get(kind, 4)


def _newer(out, src):
    return os.path.exists(out) and os.path.getmtime(out) >= os.path.getmtime(src)


def build_cpu(force=False):
    if force or not _newer(_CPU_LIB, _CPU_SRC):
        tmp = _CPU_LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               "-ffp-contract=off", "-o", tmp, _CPU_SRC, "-lm"])
        os.replace(tmp, _CPU_LIB)
    return _CPU_LIB


def build_gpu(force=False):
    if force or not _newer(_GPU_LIB, _GPU_SRC):
        tmp = _GPU_LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["hipcc", "--offload-arch=gfx950", "-O3", "-fPIC", "-shared",
                               "-ffp-contract=off",
                               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                               "-o", tmp, _GPU_SRC],
                              stderr=subprocess.DEVNULL)
        os.replace(tmp, _GPU_LIB)
    return _GPU_LIB


_cpu = None
_gpu = None


def cpu_lib():
    global _cpu
    if _cpu is None:
        # GEN_CPU_LIB names another build of gen.c to load instead (the
        # sanitizer test loads an instrumented build through it).
        path = os.environ.get("GEN_CPU_LIB") or build_cpu()
        L = ctypes.CDLL(path)
        L.gen_fill_rows_cpu.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                                        ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint64, ctypes.c_int64,
                                        ctypes.c_void_p]
        L.gen_fill_rows_cpu.restype = ctypes.c_int
        L.gen_fill_rows_list_cpu.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                                             ctypes.c_uint32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                             ctypes.c_void_p]
        L.gen_fill_rows_list_cpu.restype = ctypes.c_int
        L.gen_priorities.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int64,
                                     ctypes.c_void_p]
        L.gen_priorities.restype = ctypes.c_int
        L.gen_philox4x32_10.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.gen_philox4x32_10.restype = None
        _cpu = L
    return _cpu


def gpu_lib():
    global _gpu
    if _gpu is None:
        if not os.path.exists(_GPU_LIB):
            raise RuntimeError("gen: %s is not built (run __graft_entry__.build())" % _GPU_LIB)
        L = ctypes.CDLL(_GPU_LIB)
        L.gen_fill_rows_gpu.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                                        ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint64, ctypes.c_int64,
                                        ctypes.c_void_p, ctypes.c_void_p]
        L.gen_fill_rows_gpu.restype = ctypes.c_int
        _gpu = L
    return _gpu


def philox4x32_10(ctr, key):
    c = np.array(ctr, dtype=np.uint32)
    k = np.array(key, dtype=np.uint32)
    o = np.zeros(4, dtype=np.uint32)
    cpu_lib().gen_philox4x32_10(c.ctypes.data, k.ctypes.data, o.ctypes.data)
    return [int(x) for x in o]


@dataclass(frozen=True)
class Column:
    name: str
    kind: int
    m: int            # elements per step
    param: int = 0    # modulus for INT_MOD, reward column id for RTG_F32
    dtype: str = "u8"  # element dtype as seen by a consumer

    @property
    def elem_bytes(self):
        return self.m * elem_size(self.kind)


def fill_rows_cpu(col, col_id, seed, T, k0, nrows):
    """Rows k0..k0+nrows-1 of one column as uint8 [nrows, T*E]."""
    out = np.empty((nrows, T * col.elem_bytes), dtype=np.uint8)
    st = cpu_lib().gen_fill_rows_cpu(col.kind, col.param, col.m, seed, col_id, T, k0, nrows,
                                     out.ctypes.data)
    if st != 0:
        raise ValueError("gen_fill_rows_cpu rejected its arguments")
    return out


def fill_rows_list_cpu(col, col_id, seed, T, ks):
    """Rows of the insertions listed in ks, as uint8 [len(ks), T*E]."""
    ks = np.ascontiguousarray(ks, dtype=np.uint64)
    out = np.empty((ks.size, T * col.elem_bytes), dtype=np.uint8)
    st = cpu_lib().gen_fill_rows_list_cpu(col.kind, col.param, col.m, seed, col_id, T, ks.ctypes.data,
                                          ks.size, out.ctypes.data)
    if st != 0:
        raise ValueError("gen_fill_rows_list_cpu rejected its arguments")
    return out


def fill_rows_gpu(col, col_id, seed, T, k0, nrows, dst_ptr, stream_handle):
    """Same rows written to device (or mapped host) memory at dst_ptr."""
    st = gpu_lib().gen_fill_rows_gpu(col.kind, col.param, col.m, seed, col_id, T, k0, nrows,
                                     ctypes.c_void_p(dst_ptr), ctypes.c_void_p(stream_handle))
    if st != 0:
        raise RuntimeError("gen_fill_rows_gpu failed (%d)" % st)


@dataclass(frozen=True)
class PrioDist:
    kind: int
    a: float
    b: float
    c: float = 0.0


def priorities(dist, seed, stream, k0, n):
    out = np.empty(n, dtype=np.uint32)
    st = cpu_lib().gen_priorities(dist.kind, dist.a, dist.b, dist.c, seed, stream, k0, n,
                                  out.ctypes.data)
    if st != 0:
        raise ValueError("gen_priorities rejected its arguments")
    return out


def insert_priorities(dist, seed, k0, n):
    """Initial priorities of insertions k0..k0+n-1."""
    return priorities(dist, seed, PRIO_STREAM, k0, n)


def update_priorities(dist, seed, t, B):
    """New priorities given to the update of iteration t (one per draw)."""
    return priorities(dist, seed, UPDATE_STREAM0 + t, 0, B)


def select_seed(seed, t):
    """Seed handed to the selection of iteration t."""
    return (int(seed) << 32) + int(t)


def slot_insertion(slot, next_seq, N):
    """Insertion number held by ring slot `slot` after next_seq insertions."""
    slot = np.asarray(slot, dtype=np.int64)
    last = int(next_seq) - 1
    return slot + N * ((last - slot) // N)
