"""The oracle and the CPU input generator under AddressSanitizer and
UndefinedBehaviorSanitizer.

Both C sources are built with gcc, instrumented, into a temporary
directory, and the oracle's and generator's pins run against those builds
in a child process (ORACLE_LIB and GEN_CPU_LIB point at them; the ASan
runtime is preloaded because the Python interpreter is not instrumented).
Any out-of-bounds access, use after free or undefined operation in either
library aborts the child, which fails this test.  Nothing here runs on a
GPU, and the HIP library is not involved.
"""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = ["tests/test_oracle_rng.py", "tests/test_oracle_select.py", "tests/test_oracle_collect_update.py",
        "tests/test_oracle_allocator.py", "tests/test_golden.py", "tests/test_gen.py"]
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-std=c11", "-fPIC", "-shared", "-ffp-contract=off"]


def _runtime(name):
    return subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()


def test_oracle_and_generator_pins_under_asan_and_ubsan(tmp_path):
    orc = str(tmp_path / "liboracle_san.so")
    gen_lib = str(tmp_path / "libgen_san.so")
    subprocess.run(["gcc"] + SAN + ["-o", orc, os.path.join(ROOT, "oracle", "oracle.c"), "-lm"], check=True)
    subprocess.run(["gcc"] + SAN + ["-fopenmp", "-o", gen_lib, os.path.join(ROOT, "gen", "gen.c"), "-lm"], check=True)
    env = dict(os.environ, ORACLE_LIB=orc, GEN_CPU_LIB=gen_lib, PYTHONDONTWRITEBYTECODE="1",
               LD_PRELOAD=_runtime("libasan.so"),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider"] + PINS,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout[-3000:] + r.stderr[-3000:]
    assert r.returncode == 0, out
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out
    # The child really loaded the instrumented builds.
    probe = ("import oracle, gen; print(oracle.lib()._name); print(gen.cpu_lib()._name)")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr[-2000:]
    assert r.stdout.split() == [orc, gen_lib]
