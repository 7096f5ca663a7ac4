"""Host-side logic of bench.py that needs no GPU: it refuses more than one
GPU, and it reports gather traffic only from a counter summary taken on the
current gather source."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_traffic_comes_from_a_summary_of_the_current_source(tmp_path, monkeypatch):
    sha = bench.source_sha(bench.GATHER_SRC)
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    summary = "# comment: 1\nkernel: collect_kernel\nsource_sha256: %s\ntraffic_bytes_per_launch: 12345\n"
    (prof / "gather_mat_counters.txt").write_text(summary % sha)
    assert bench.profiled_traffic("collect_kernel", "mat") == 12345.0
    # Taken on another version of the gather: no traffic figure.
    (prof / "gather_mat_counters.txt").write_text(summary % ("0" * 64))
    assert bench.profiled_traffic("collect_kernel", "mat") is None
    # Another kernel, or no summary at all: none either.
    (prof / "gather_mat_counters.txt").write_text(summary % sha)
    assert bench.profiled_traffic("other_kernel", "mat") is None
    assert bench.profiled_traffic("collect_kernel", "dt") is None

