"""Python binding of libgear.so (the C ABI declared in include/gear.h).

Each ``gear_*`` function here has the name and meaning of the C entry point
and only marshals arguments: pointers are Python ints (a torch tensor's
``data_ptr()``), streams are ``hipStream_t`` handles as ints (torch's
``cuda_stream``; 0 is the null stream).  Every step of the hot path runs in
the HIP library; a failing call raises ``GearError``.  ``Table`` is a
convenience wrapper that takes torch tensors and uses torch only to allocate
device memory and to name the current stream.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libgear.so")

GEAR_OK = 0
GEAR_E_INVAL = -1
GEAR_E_NOMEM = -2
GEAR_E_EMPTY = -3
GEAR_E_INSUFFICIENT = -4
GEAR_E_HIP = -5
GEAR_STATUS_NO_WEIGHT = 1
GEAR_STATUS_BAD_INDEX = 2
GEAR_STATUS_INTERNAL = 4
GEAR_DEVICE = 0
GEAR_HOST_PINNED = 1
GEAR_FIFO = 0
GEAR_LIFO = 1
GEAR_UNIFORM = 2
GEAR_PRIORITIZED = 3
GEAR_TOPK = 4
GEAR_MAX_CAPACITY = 1 << 30
GEAR_MAX_COLUMNS = 64
GEAR_MAX_BATCH = 1 << 24
GEAR_MAX_TOPK = 16384
GEAR_NOALLOC_MAX_N = 1 << 24
GEAR_NOALLOC_SCRATCH_BYTES = 536832
GEAR_SMALL_SELECT_MAX_N = 16384
GEAR_SMALL_SELECT_MAX_B = 2048
GEAR_OPT_INCREMENTAL_TREE = 1
GEAR_OPT_IS_GLOBAL_MIN = 2
GEAR_OPT_GATHER_SHARE_CU = 4
GEAR_DTYPE_U8, GEAR_DTYPE_I8, GEAR_DTYPE_U16, GEAR_DTYPE_I16, GEAR_DTYPE_F16, GEAR_DTYPE_BF16 = 0, 1, 2, 3, 4, 5
GEAR_DTYPE_U32, GEAR_DTYPE_I32, GEAR_DTYPE_F32, GEAR_DTYPE_U64, GEAR_DTYPE_I64, GEAR_DTYPE_F64 = 6, 7, 8, 9, 10, 11
GEAR_MAX_NAME = 63
# torch dtype name of each GEAR_DTYPE_* (the library only moves bytes).
DTYPE_NAMES = {GEAR_DTYPE_U8: "uint8", GEAR_DTYPE_I8: "int8", GEAR_DTYPE_U16: "uint16", GEAR_DTYPE_I16: "int16",
               GEAR_DTYPE_F16: "float16", GEAR_DTYPE_BF16: "bfloat16", GEAR_DTYPE_U32: "uint32",
               GEAR_DTYPE_I32: "int32", GEAR_DTYPE_F32: "float32", GEAR_DTYPE_U64: "uint64", GEAR_DTYPE_I64: "int64",
               GEAR_DTYPE_F64: "float64"}
DTYPE_BYTES = {GEAR_DTYPE_U8: 1, GEAR_DTYPE_I8: 1, GEAR_DTYPE_U16: 2, GEAR_DTYPE_I16: 2, GEAR_DTYPE_F16: 2,
               GEAR_DTYPE_BF16: 2, GEAR_DTYPE_U32: 4, GEAR_DTYPE_I32: 4, GEAR_DTYPE_F32: 4, GEAR_DTYPE_U64: 8,
               GEAR_DTYPE_I64: 8, GEAR_DTYPE_F64: 8}


class gear_column(ctypes.Structure):
    """Mirror of the C descriptor gear_column."""
    _fields_ = [("name", ctypes.c_char_p), ("dtype", ctypes.c_int32), ("elems_per_step", ctypes.c_int32)]


class GearError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("%s (code %d)" % (msg, code))
        self.code = code


_lib = None


def lib():
    """The loaded libgear.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libgear.so is not built at %s: run __graft_entry__.build() "
                               "or python -m paper_2310_05205_amd.build" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
        L.gear_table_create.argtypes = [vp, i32, i64, i32, i32, i32, ctypes.POINTER(vp)]
        L.gear_table_destroy.argtypes = [vp]
        L.gear_insert.argtypes = [vp, i64, vp, vp, vp]
        L.gear_select.argtypes = [vp, i32, i32, i32, u64, ctypes.c_float, vp, vp, vp, vp]
        L.gear_collect.argtypes = [vp, vp, vp, i32, i32, vp, i32, vp, vp]
        L.gear_select_collect.argtypes = [vp, i32, i32, i32, u64, vp, vp, vp, vp, i32, vp, vp]
        L.gear_update_priorities.argtypes = [vp, vp, vp, i32, vp]
        L.gear_table_sync.argtypes = [vp, vp, ctypes.POINTER(i32)]
        L.gear_table_info.argtypes = [vp, ctypes.POINTER(i64), ctypes.POINTER(u64)]
        L.gear_table_column.argtypes = [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(i64)]
        L.gear_table_priorities.argtypes = [vp, ctypes.POINTER(vp)]
        L.gear_table_set_options.argtypes = [vp, ctypes.c_uint32]
        L.gear_table_use_allocator.argtypes = [vp, i32, i64]
        L.gear_allocate.argtypes = [vp, i64, vp, vp]
        L.gear_commit.argtypes = [vp, i64, vp, vp, vp]
        pi64 = ctypes.POINTER(i64)
        L.gear_allocator_info.argtypes = [vp, pi64, pi64, pi64]
        L.gear_write_rows.argtypes = [vp, i64, vp, vp, vp]
        L.gear_shard_total.argtypes = [vp, vp, vp]
        L.gear_select_shard.argtypes = [vp, i32, i32, vp, i64, i32, i32, u64, vp, vp, vp, vp]
        L.gear_is_weights.argtypes = [vp, vp, i32, ctypes.c_float, vp, vp]
        L.gear_topk_merge.argtypes = [vp, vp, i32, i32, i32, i32, u64, vp, vp, vp, vp, vp]
        L.gear_select_prioritized_noalloc.argtypes = [vp, i64, i32, i32, i32, u64, ctypes.c_float, vp, vp, vp, vp]
        L.gear_table_create_columns.argtypes = [ctypes.POINTER(gear_column), i32, i64, i32, i32, i32,
                                                ctypes.POINTER(vp)]
        L.gear_table_column_info.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(i32),
                                             ctypes.POINTER(i32)]
        L.gear_table_find_column.argtypes = [vp, ctypes.c_char_p, ctypes.POINTER(i32)]
        for name in ["gear_table_create", "gear_table_destroy", "gear_insert", "gear_select", "gear_collect",
                     "gear_select_collect",
                     "gear_update_priorities", "gear_table_sync", "gear_table_info", "gear_table_column",
                     "gear_table_priorities", "gear_table_set_options", "gear_table_use_allocator",
                     "gear_allocate", "gear_commit", "gear_allocator_info", "gear_write_rows", "gear_shard_total",
                     "gear_select_shard", "gear_is_weights", "gear_topk_merge",
                     "gear_select_prioritized_noalloc", "gear_table_create_columns", "gear_table_column_info",
                     "gear_table_find_column"]:
            getattr(L, name).restype = ctypes.c_int
        L.gear_last_error.argtypes = []
        L.gear_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def gear_last_error():
    return lib().gear_last_error().decode()


def _check(code):
    if code != GEAR_OK:
        raise GearError(code, gear_last_error())
    return code


def _ptr_array(ptrs):
    arr = (ctypes.c_void_p * max(len(ptrs), 1))()
    for i, p in enumerate(ptrs):
        arr[i] = p
    return arr


def gear_table_create(elem_bytes, capacity, T, residency=GEAR_DEVICE, device=0):
    eb = (ctypes.c_int64 * max(len(elem_bytes), 1))(*[int(e) for e in elem_bytes])
    out = ctypes.c_void_p()
    _check(lib().gear_table_create(eb, len(elem_bytes), int(capacity), int(T), int(residency), int(device),
                                   ctypes.byref(out)))
    return out.value


def gear_table_create_columns(columns, capacity, T, residency=GEAR_DEVICE, device=0):
    """columns: list of (name, GEAR_DTYPE_*, elems_per_step)."""
    arr = (gear_column * max(len(columns), 1))()
    keep = []
    for i, (name, dtype, elems) in enumerate(columns):
        b = name.encode()
        keep.append(b)
        arr[i] = gear_column(b, int(dtype), int(elems))
    out = ctypes.c_void_p()
    _check(lib().gear_table_create_columns(arr, len(columns), int(capacity), int(T), int(residency), int(device),
                                           ctypes.byref(out)))
    return out.value


def gear_table_column_info(table, c):
    name = ctypes.c_char_p()
    dtype, elems = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().gear_table_column_info(table, int(c), ctypes.byref(name), ctypes.byref(dtype), ctypes.byref(elems)))
    return name.value.decode(), dtype.value, elems.value


def gear_table_find_column(table, name):
    c = ctypes.c_int32(-1)
    _check(lib().gear_table_find_column(table, name.encode(), ctypes.byref(c)))
    return c.value


def gear_table_destroy(table):
    _check(lib().gear_table_destroy(table))


def gear_insert(table, n, col_src, priorities, stream=0):
    """col_src: list of pointers (host or device), priorities: pointer."""
    arr = _ptr_array(col_src) if col_src is not None else None
    _check(lib().gear_insert(table, int(n), arr, priorities, stream))


def gear_select(table, strategy, B, L, seed, beta, d_idx, d_start, d_weights=0, stream=0):
    _check(lib().gear_select(table, int(strategy), int(B), int(L), int(seed) & ((1 << 64) - 1),
                             ctypes.c_float(beta), d_idx, d_start, d_weights or None, stream))


def gear_select_prioritized_noalloc(d_priority, N, T, B, L, seed, beta, d_idx, d_start, d_weights=0, stream=0):
    _check(lib().gear_select_prioritized_noalloc(d_priority, int(N), int(T), int(B), int(L),
                                                 int(seed) & ((1 << 64) - 1), ctypes.c_float(beta), d_idx, d_start,
                                                 d_weights or None, stream))


def gear_collect(table, d_idx, d_start, B, L, col_ids, d_out, stream=0):
    """col_ids: list of column numbers or None (all); d_out: list of device pointers."""
    ids = (ctypes.c_int32 * len(col_ids))(*col_ids) if col_ids is not None else None
    _check(lib().gear_collect(table, d_idx, d_start, int(B), int(L), ids, len(d_out), _ptr_array(d_out), stream))


def gear_select_collect(table, strategy, B, L, seed, d_idx, d_start, d_weights, col_ids, d_out, stream=0):
    """FIFO, LIFO or uniform selection and the gather of its windows in one
    launch; col_ids: list of column numbers or None (all)."""
    ids = (ctypes.c_int32 * len(col_ids))(*col_ids) if col_ids is not None else None
    _check(lib().gear_select_collect(table, int(strategy), int(B), int(L), int(seed) & ((1 << 64) - 1), d_idx,
                                     d_start, d_weights or None, ids, len(d_out), _ptr_array(d_out), stream))


def gear_update_priorities(table, d_idx, d_new_priorities, B, stream=0):
    _check(lib().gear_update_priorities(table, d_idx, d_new_priorities, int(B), stream))


def gear_table_sync(table, stream=0):
    st = ctypes.c_int32(0)
    _check(lib().gear_table_sync(table, stream, ctypes.byref(st)))
    return st.value


def gear_table_info(table):
    count = ctypes.c_int64(0)
    nseq = ctypes.c_uint64(0)
    _check(lib().gear_table_info(table, ctypes.byref(count), ctypes.byref(nseq)))
    return count.value, nseq.value


def gear_table_column(table, c):
    base = ctypes.c_void_p()
    host = ctypes.c_void_p()
    eb = ctypes.c_int64(0)
    _check(lib().gear_table_column(table, int(c), ctypes.byref(base), ctypes.byref(host), ctypes.byref(eb)))
    return base.value, host.value, eb.value


def gear_table_set_options(table, options):
    _check(lib().gear_table_set_options(table, int(options)))


def gear_table_priorities(table):
    p = ctypes.c_void_p()
    _check(lib().gear_table_priorities(table, ctypes.byref(p)))
    return p.value


def gear_table_use_allocator(table, removal, max_selectable):
    _check(lib().gear_table_use_allocator(table, int(removal), int(max_selectable)))


def gear_allocate(table, n, stream=0):
    """Returns the n allocated indices as a host int64 numpy array."""
    import numpy as np
    idx = np.zeros(max(int(n), 1), dtype=np.int64)
    _check(lib().gear_allocate(table, int(n), idx.ctypes.data, stream))
    return idx[:int(n)]


def gear_commit(table, idx, priorities, stream=0):
    """idx: host int64 numpy array; priorities: pointer (host or device)."""
    import numpy as np
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    _check(lib().gear_commit(table, idx.size, idx.ctypes.data, priorities, stream))


def gear_write_rows(table, idx, col_src, stream=0):
    """idx: host int64 numpy array; col_src: list of pointers (host or device)."""
    import numpy as np
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    _check(lib().gear_write_rows(table, idx.size, idx.ctypes.data, _ptr_array(col_src), stream))


def gear_allocator_info(table):
    c, p, f = ctypes.c_int64(0), ctypes.c_int64(0), ctypes.c_int64(0)
    _check(lib().gear_allocator_info(table, ctypes.byref(c), ctypes.byref(p), ctypes.byref(f)))
    return c.value, p.value, f.value


def gear_shard_total(table, d_total, stream=0):
    _check(lib().gear_shard_total(table, d_total, stream))


def gear_select_shard(table, G, g, d_totals, base, B, L, seed, d_idx, d_start, d_sel_prio=0, stream=0):
    _check(lib().gear_select_shard(table, int(G), int(g), d_totals, int(base), int(B), int(L),
                                   int(seed) & ((1 << 64) - 1), d_idx, d_start, d_sel_prio or None, stream))


def gear_is_weights(table, d_sel_prio, B, beta, d_weights, stream=0):
    _check(lib().gear_is_weights(table, d_sel_prio, int(B), ctypes.c_float(beta), d_weights, stream))


def gear_topk_merge(d_prio, d_gidx, G, K, T, L, seed, d_idx, d_start, d_weights=0, d_out_prio=0, stream=0):
    _check(lib().gear_topk_merge(d_prio, d_gidx, int(G), int(K), int(T), int(L), int(seed) & ((1 << 64) - 1),
                                 d_idx, d_start, d_weights or None, d_out_prio or None, stream))


def topk_merge(prio, gidx, K, T, L, seed, device=0):
    """Global top-K of G sorted local top-K lists (torch tensors [G, K] of
    uint32-valued priorities and int64 global indices on `device`).
    Returns (idx, start, weights, priorities)."""
    import torch
    dev = torch.device("cuda", device)
    G = int(gidx.shape[0])
    idx = torch.empty(K, dtype=torch.int64, device=dev)
    start = torch.empty(K, dtype=torch.int32, device=dev)
    w = torch.empty(K, dtype=torch.float32, device=dev)
    p = torch.empty(K, dtype=torch.int32, device=dev)
    prio = prio.contiguous()
    gidx = gidx.contiguous()
    gear_topk_merge(prio.data_ptr(), gidx.data_ptr(), G, K, T, L, seed, idx.data_ptr(), start.data_ptr(),
                    w.data_ptr(), p.data_ptr(), torch.cuda.current_stream(dev).cuda_stream)
    return idx, start, w, p


class _DeviceBytes:
    """Describes device memory to torch.as_tensor (array-interface protocol)."""

    def __init__(self, ptr, shape):
        self.__cuda_array_interface__ = {"shape": tuple(shape), "typestr": "|u1", "data": (int(ptr), False),
                                         "strides": None, "version": 2}


def _dtype_code(dtype):
    """GEAR_DTYPE_* of a torch dtype, a dtype name ("bfloat16", "bf16", ...) or a code."""
    if isinstance(dtype, int):
        return dtype
    name = str(dtype).replace("torch.", "")
    alias = {"u8": "uint8", "i8": "int8", "u16": "uint16", "i16": "int16", "f16": "float16", "half": "float16",
             "bf16": "bfloat16", "u32": "uint32", "i32": "int32", "f32": "float32", "float": "float32",
             "u64": "uint64", "i64": "int64", "f64": "float64", "double": "float64"}
    name = alias.get(name, name)
    for code, n in DTYPE_NAMES.items():
        if n == name:
            return code
    raise ValueError("no GEAR dtype for %r" % (dtype,))


class ColumnSpec:
    """One typed column: name, GEAR_DTYPE_* code, per-step shape."""

    def __init__(self, name, dtype, shape):
        self.name = str(name)
        self.dtype = _dtype_code(dtype)
        self.shape = tuple(int(x) for x in shape)
        n = 1
        for x in self.shape:
            n *= x
        self.elems = n
        self.elem_bytes = n * DTYPE_BYTES[self.dtype]

    def torch_dtype(self):
        import torch
        return getattr(torch, DTYPE_NAMES[self.dtype])


class Table:
    """A replay store over torch tensors.

    ``columns`` is a list of bytes-per-step sizes (byte columns), or of typed
    columns: (name, dtype, per-step shape) tuples or ColumnSpec objects, or a
    dict {name: (dtype, shape)}.  Outputs are allocated as torch CUDA tensors
    on the table's device; work is issued on torch's current stream of that
    device.
    """

    def __init__(self, columns, capacity, T, residency=GEAR_DEVICE, device=0):
        import torch
        self._torch = torch
        if isinstance(columns, dict):
            columns = [(name, spec[0], spec[1]) for name, spec in columns.items()]
        columns = list(columns)
        self.capacity, self.T, self.device = int(capacity), int(T), int(device)
        self.residency = residency
        typed = not all(isinstance(c, int) for c in columns)
        if typed:
            specs = [c if isinstance(c, ColumnSpec) else ColumnSpec(*c) for c in columns]
            self.elem_bytes = [c.elem_bytes for c in specs]
            self.handle = gear_table_create_columns([(c.name, c.dtype, c.elems) for c in specs], capacity, T,
                                                    residency, device)
        else:
            self.elem_bytes = [int(e) for e in columns]
            self.handle = gear_table_create(self.elem_bytes, capacity, T, residency, device)
        # Names, types and shapes as the library keeps them (byte columns:
        # "c<index>", uint8, shape (elem_bytes,)); typed specs keep their shape.
        self.columns = []
        for c in range(len(self.elem_bytes)):
            name, dtype, elems = gear_table_column_info(self.handle, c)
            self.columns.append(ColumnSpec(name, dtype, specs[c].shape if typed else (elems,)))
        self._index = {c.name: i for i, c in enumerate(self.columns)}

    def close(self):
        if self.handle:
            gear_table_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _stream(self, stream):
        if stream is not None:
            return stream.cuda_stream
        return self._torch.cuda.current_stream(self.device).cuda_stream

    def _sources(self, col_src):
        """Pointers of the column sources, in column order: a list, or a dict
        keyed by column name (every column; contiguous tensors or arrays)."""
        if isinstance(col_src, dict):
            missing = [c.name for c in self.columns if c.name not in col_src]
            if missing:
                raise ValueError("no source for columns %s" % missing)
            col_src = [col_src[c.name] for c in self.columns]
        for x in col_src:
            if hasattr(x, "is_contiguous") and not x.is_contiguous():
                raise ValueError("column sources must be contiguous")
        return [_data_ptr(x) for x in col_src]

    def insert(self, col_src, priorities, stream=None):
        """col_src: per column, [n, T, *shape] data ([n, T*E_c] bytes for byte
        columns), host or device, as a list in column order or a dict keyed by
        name; priorities uint32[n]."""
        n = int(priorities.shape[0])
        gear_insert(self.handle, n, self._sources(col_src), _data_ptr(priorities), self._stream(stream))

    def select(self, strategy, B, L, seed, beta=0.0, weights=False, stream=None):
        torch = self._torch
        dev = torch.device("cuda", self.device)
        idx = torch.empty(B, dtype=torch.int64, device=dev)
        start = torch.empty(B, dtype=torch.int32, device=dev)
        w = torch.empty(B, dtype=torch.float32, device=dev) if weights else None
        gear_select(self.handle, strategy, B, L, seed, beta, idx.data_ptr(), start.data_ptr(),
                    w.data_ptr() if w is not None else 0, self._stream(stream))
        return idx, start, w

    def collect(self, idx, start, L, col_ids=None, stream=None, out=None):
        """Returns a list of uint8 tensors [B, L*E_c], one per requested column."""
        torch = self._torch
        B = int(idx.shape[0])
        cols = list(range(len(self.elem_bytes))) if col_ids is None else list(col_ids)
        if out is None:
            dev = torch.device("cuda", self.device)
            out = [torch.empty((B, L * self.elem_bytes[c]), dtype=torch.uint8, device=dev) for c in cols]
        gear_collect(self.handle, idx.data_ptr(), start.data_ptr(), B, L, col_ids,
                     [o.data_ptr() for o in out], self._stream(stream))
        return out

    def select_collect_fields(self, strategy, B, L, seed, fields=None, weights=False, stream=None):
        """select_collect with the batch as {name: tensor[B, L, *shape]} views
        of each column's dtype, as collect_fields returns them."""
        names = [c.name for c in self.columns] if fields is None else list(fields)
        ids = [self._index[n] for n in names]
        idx, start, w, raw = self.select_collect(strategy, B, L, seed, weights=weights, col_ids=ids, stream=stream)
        res = {}
        for n, c, r in zip(names, ids, raw):
            spec = self.columns[c]
            res[n] = r.view(spec.torch_dtype()).view((B, L) + spec.shape)
        return idx, start, w, res

    def select_collect(self, strategy, B, L, seed, weights=False, col_ids=None, stream=None):
        """FIFO, LIFO or uniform selection and its gather in one launch:
        (idx, start, w, list of uint8 tensors [B, L*E_c]), equal to select()
        followed by collect()."""
        torch = self._torch
        dev = torch.device("cuda", self.device)
        idx = torch.empty(B, dtype=torch.int64, device=dev)
        start = torch.empty(B, dtype=torch.int32, device=dev)
        w = torch.empty(B, dtype=torch.float32, device=dev) if weights else None
        cols = list(range(len(self.elem_bytes))) if col_ids is None else list(col_ids)
        out = [torch.empty((B, L * self.elem_bytes[c]), dtype=torch.uint8, device=dev) for c in cols]
        gear_select_collect(self.handle, strategy, B, L, seed, idx.data_ptr(), start.data_ptr(),
                            w.data_ptr() if w is not None else 0, col_ids, [o.data_ptr() for o in out],
                            self._stream(stream))
        return idx, start, w, out

    def collect_fields(self, idx, start, L, fields=None, stream=None, out=None):
        """The batch as {name: tensor[B, L, *shape]} of each column's dtype
        (Sec. 3.4: collect(indices, fields) handed over as tensors).  The
        tensors are views of the byte batches that gear_collect writes (no
        copy, no arithmetic); `out`, if given, is the dict of byte buffers
        [B, L*E] to reuse."""
        names = [c.name for c in self.columns] if fields is None else list(fields)
        ids = [self._index[n] for n in names]
        raw = self.collect(idx, start, L, col_ids=ids, stream=stream,
                           out=None if out is None else [out[n] for n in names])
        B = int(idx.shape[0])
        res = {}
        for n, c, r in zip(names, ids, raw):
            spec = self.columns[c]
            res[n] = r.view(spec.torch_dtype()).view((B, L) + spec.shape)
        return res

    def column_index(self, name):
        return gear_table_find_column(self.handle, name)

    def update_priorities(self, idx, new_priorities, stream=None):
        gear_update_priorities(self.handle, idx.data_ptr(), new_priorities.data_ptr(), int(idx.shape[0]),
                               self._stream(stream))

    def set_options(self, options):
        gear_table_set_options(self.handle, options)

    def use_allocator(self, removal, max_selectable=None):
        """Switch to allocate/commit insertion with FIFO or LIFO removal."""
        gear_table_use_allocator(self.handle, removal, self.capacity if max_selectable is None else max_selectable)

    def allocate(self, n, stream=None):
        """n free indices (host int64 array); victims are released on the stream."""
        return gear_allocate(self.handle, n, self._stream(stream))

    def commit(self, idx, priorities, stream=None):
        """Commit pending indices (host int64) with uint32 priorities (host or device)."""
        gear_commit(self.handle, idx, _data_ptr(priorities), self._stream(stream))

    def allocator_info(self):
        return gear_allocator_info(self.handle)

    def write_rows(self, idx, col_src, stream=None):
        """Write row r of each column source ([n, T, *shape] per column, a list
        or a dict keyed by name) into slot idx[r]."""
        gear_write_rows(self.handle, idx, self._sources(col_src), self._stream(stream))

    def shard_total(self, out, stream=None):
        """Writes this table's priority total into `out` (a one-element int64
        or uint64-sized device tensor view)."""
        gear_shard_total(self.handle, out.data_ptr(), self._stream(stream))

    def select_shard(self, G, g, totals, base, B, L, seed, stream=None):
        """Shard g's part of prioritized selection; returns (idx, start, sel_prio)."""
        torch = self._torch
        dev = torch.device("cuda", self.device)
        idx = torch.empty(B, dtype=torch.int64, device=dev)
        start = torch.empty(B, dtype=torch.int32, device=dev)
        p = torch.empty(B, dtype=torch.int32, device=dev)
        gear_select_shard(self.handle, G, g, totals.data_ptr(), base, B, L, seed, idx.data_ptr(), start.data_ptr(),
                          p.data_ptr(), self._stream(stream))
        return idx, start, p

    def is_weights(self, sel_prio, beta, stream=None):
        torch = self._torch
        w = torch.empty(int(sel_prio.shape[0]), dtype=torch.float32, device=torch.device("cuda", self.device))
        gear_is_weights(self.handle, sel_prio.data_ptr(), int(sel_prio.shape[0]), beta, w.data_ptr(),
                        self._stream(stream))
        return w

    def column_view(self, c):
        """Column c's blocks in place, [capacity, T*E_c] bytes: a torch uint8
        tensor over the table's HBM (device tables) or a numpy array over its
        pinned host memory.  Writing rows of allocated indices through it is
        the in-place insertion path; the view must not outlive the table."""
        import numpy as np
        base, host, eb = gear_table_column(self.handle, c)
        shape = (self.capacity, self.T * eb)
        if self.residency == GEAR_HOST_PINNED:
            buf = (ctypes.c_uint8 * (shape[0] * shape[1])).from_address(host)
            return np.ctypeslib.as_array(buf).reshape(shape)
        torch = self._torch
        return torch.as_tensor(_DeviceBytes(base, shape), device=torch.device("cuda", self.device))

    def sync(self, stream=None):
        return gear_table_sync(self.handle, self._stream(stream))

    def info(self):
        return gear_table_info(self.handle)

    def priorities(self):
        """Copy of the priority array as a CPU uint32 numpy array."""
        import numpy as np
        torch = self._torch
        ptr = gear_table_priorities(self.handle)
        host = np.empty(self.capacity, dtype=np.uint32)
        torch.cuda.synchronize(self.device)
        _hip_memcpy_d2h(host.ctypes.data, ptr, host.nbytes)
        return host


def _data_ptr(x):
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    return x.ctypes.data


_hip = None


def _hip_memcpy_d2h(dst, src, nbytes):
    """Plain hipMemcpy for reading table state back (tests, checks)."""
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime libgear.so is bound to
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        _hip.hipMemcpy.restype = ctypes.c_int
    rc = _hip.hipMemcpy(dst, src, nbytes, 2)  # hipMemcpyDeviceToHost
    if rc != 0:
        raise RuntimeError("hipMemcpy failed (%d)" % rc)
