"""CPU checks of the C ABI: the library loads, exports every function that
include/gear.h declares, and rejects invalid arguments before touching a
device.  No compute call is made here."""
import ctypes
import os
import re

import pytest

from paper_2310_05205_amd import gear

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "gear.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gear_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert "gear_select" in names and "gear_collect" in names and len(names) >= 10
    lib = gear.lib()
    for n in names:
        assert hasattr(lib, n), n


def test_every_exported_symbol_is_declared():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", gear.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (gear_[a-z_]+)$", out, flags=re.M))
    assert exported and exported <= set(_declared()), sorted(exported - set(_declared()))


def test_header_constants_match_binding():
    with open(os.path.join(ROOT, "include", "gear.h")) as f:
        text = f.read()
    for name, val in re.findall(r"#define (GEAR_[A-Z_]+)\s+(-?\d+)u?\b", text):
        if hasattr(gear, name):
            assert getattr(gear, name) == int(val), name


def test_argument_validation_without_device():
    lib = gear.lib()
    out = ctypes.c_void_p()
    eb = (ctypes.c_int64 * 1)(4)
    assert lib.gear_table_create(eb, 1, 16, 4, 0, 0, None) == gear.GEAR_E_INVAL
    assert lib.gear_table_create(eb, 1, 0, 4, 0, 0, ctypes.byref(out)) == gear.GEAR_E_INVAL
    assert lib.gear_table_create(eb, 1, 16, 0, 0, 0, ctypes.byref(out)) == gear.GEAR_E_INVAL
    assert lib.gear_table_create(eb, 1, 16, 4, 7, 0, ctypes.byref(out)) == gear.GEAR_E_INVAL
    assert lib.gear_table_create(eb, -1, 16, 4, 0, 0, ctypes.byref(out)) == gear.GEAR_E_INVAL
    assert lib.gear_table_create(None, 1, 16, 4, 0, 0, ctypes.byref(out)) == gear.GEAR_E_INVAL
    assert lib.gear_table_create(eb, 1, (1 << 30) + 1, 4, 0, 0, ctypes.byref(out)) == gear.GEAR_E_INVAL
    assert "capacity" in gear.gear_last_error()
    assert lib.gear_select(None, 3, 1, 1, 0, ctypes.c_float(0), None, None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_collect(None, None, None, 1, 1, None, 1, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_select_collect(None, 0, 1, 1, 0, None, None, None, None, 1, None, None) == gear.GEAR_E_INVAL
    assert "gear_select_collect" in gear.gear_last_error()
    assert lib.gear_update_priorities(None, None, None, 1, None) == gear.GEAR_E_INVAL
    assert lib.gear_insert(None, 1, None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_table_sync(None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_table_info(None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_table_destroy(None) == gear.GEAR_OK
    assert lib.gear_table_use_allocator(None, 0, 1) == gear.GEAR_E_INVAL
    assert lib.gear_allocate(None, 1, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_commit(None, 1, None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_allocator_info(None, None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_shard_total(None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_write_rows(None, 1, None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_select_shard(None, 1, 0, None, 0, 1, 1, 0, None, None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_is_weights(None, None, 1, ctypes.c_float(0), None, None) == gear.GEAR_E_INVAL
    assert lib.gear_topk_merge(None, None, 0, 1, 1, 1, 0, None, None, None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_topk_merge(None, None, 2, 1, 1, 1, 0, None, None, None, None, None) == gear.GEAR_E_INVAL
    f0 = ctypes.c_float(0)
    assert lib.gear_select_prioritized_noalloc(None, 16, 4, 4, 1, 0, f0, None, None, None, None) == gear.GEAR_E_INVAL
    assert lib.gear_select_prioritized_noalloc(16, gear.GEAR_NOALLOC_MAX_N + 1, 4, 4, 1, 0, f0, 16, 16, None,
                                               None) == gear.GEAR_E_INVAL
    assert "GEAR_NOALLOC_MAX_N" in gear.gear_last_error()
    with pytest.raises(gear.GearError) as e:
        gear.gear_table_create([4], 16, 0)
    assert e.value.code == gear.GEAR_E_INVAL


def test_typed_column_descriptors_are_validated_without_device():
    lib = gear.lib()
    out = ctypes.c_void_p()

    def create(cols):
        arr = (gear.gear_column * max(len(cols), 1))(*[gear.gear_column(n, d, e) for n, d, e in cols])
        return lib.gear_table_create_columns(arr, len(cols), 16, 4, 0, 0, ctypes.byref(out))

    assert create([(None, gear.GEAR_DTYPE_F32, 1)]) == gear.GEAR_E_INVAL
    assert "NULL" in gear.gear_last_error()
    assert create([(b"", gear.GEAR_DTYPE_F32, 1)]) == gear.GEAR_E_INVAL
    assert create([(b"x" * (gear.GEAR_MAX_NAME + 1), gear.GEAR_DTYPE_F32, 1)]) == gear.GEAR_E_INVAL
    assert create([(b"obs", gear.GEAR_DTYPE_F32, 1), (b"obs", gear.GEAR_DTYPE_I32, 2)]) == gear.GEAR_E_INVAL
    assert "repeated" in gear.gear_last_error()
    assert create([(b"obs", 12, 1)]) == gear.GEAR_E_INVAL
    assert create([(b"obs", -1, 1)]) == gear.GEAR_E_INVAL
    assert create([(b"obs", gear.GEAR_DTYPE_BF16, 0)]) == gear.GEAR_E_INVAL
    assert lib.gear_table_create_columns(None, 1, 16, 4, 0, 0, ctypes.byref(out)) == gear.GEAR_E_INVAL
    assert lib.gear_table_create_columns(None, 0, 16, 4, 0, 0, None) == gear.GEAR_E_INVAL
    c = ctypes.c_int32(5)
    assert lib.gear_table_find_column(None, b"obs", ctypes.byref(c)) == gear.GEAR_E_INVAL and c.value == -1
    assert lib.gear_table_column_info(None, 0, None, None, None) == gear.GEAR_E_INVAL


def test_column_specs_map_torch_dtypes():
    spec = gear.ColumnSpec("obs", "bfloat16", (8, 64))
    assert spec.dtype == gear.GEAR_DTYPE_BF16 and spec.elems == 512 and spec.elem_bytes == 1024
    assert gear.ColumnSpec("a", "i32", (8,)).elem_bytes == 32
    assert gear.ColumnSpec("r", "float32", ()).elem_bytes == 4
    for code, name in gear.DTYPE_NAMES.items():
        assert gear._dtype_code(name) == code and gear._dtype_code("torch." + name) == code
    with pytest.raises(ValueError):
        gear._dtype_code("complex64")


def test_product_has_no_oracle_or_fallback():
    """The product package must not reach the oracle or a CPU path."""
    pkg = os.path.join(ROOT, "paper_2310_05205_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".h", ".cpp")):
                with open(os.path.join(dirpath, fn)) as f:
                    src = f.read()
                assert "import oracle" not in src and "from oracle" not in src, fn
                assert "oracle_" not in src, fn


def test_missing_library_fails_loudly():
    """Without a built libgear.so the binding raises; there is no fallback."""
    from paper_2310_05205_amd import gear
    saved_path, saved_lib = gear.LIB_PATH, gear._lib
    try:
        gear.LIB_PATH = os.path.join(ROOT, "_no_such_dir", "libgear.so")
        gear._lib = None
        with pytest.raises(RuntimeError, match="not built"):
            gear.lib()
        with pytest.raises(RuntimeError, match="not built"):
            gear.gear_table_create([4], 16, 2)
    finally:
        gear.LIB_PATH, gear._lib = saved_path, saved_lib
