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



def test_pipeline_groups_ramp_then_fixed_size():
    assert bench.pipeline_groups(0, 4) == []
    assert [len(g) for g in bench.pipeline_groups(20, 4)] == [1, 2, 4, 4, 4, 4, 1]
    assert [len(g) for g in bench.pipeline_groups(5, 4)] == [1, 2, 2]
    assert [len(g) for g in bench.pipeline_groups(6, 1)] == [1] * 6
    for group in range(1, 9):
        for n in range(0, 41):
            gl = bench.pipeline_groups(n, group)
            assert [j for g in gl for j in g] == list(range(n))
            assert all(1 <= len(g) <= group for g in gl)


def test_buffer_sets_are_not_rewritten_before_their_gathers_end():
    """The selection stream writes a step's set only after the gather stream
    has finished every earlier group that used that set (gathers run in
    order, so waiting for a group covers the groups before it).  With
    2*group sets it never waits for the group just before, which the gather
    stream is still running while the next group is selected."""
    for group in range(1, 9):
        nsets = 2 * group
        for n in range(0, 60):
            gl = bench.pipeline_groups(n, group)
            waits = bench.set_reuse_waits(gl, nsets)
            assert len(waits) == len(gl)
            seen = -1      # latest group the selection stream has waited for
            last = {}
            for g, (js, ws) in enumerate(zip(gl, waits)):
                assert len({j % nsets for j in js}) == len(js)
                seen = max([seen] + ws)
                for j in js:
                    assert last.get(j % nsets, -1) <= seen
                assert g - 1 not in ws
                for j in js:
                    last[j % nsets] = g


def test_graph_mode_only_for_steps_whose_captures_replay():
    from gen import configs
    from paper_2310_05205_amd import gear
    assert bench.capturable(configs.DT, 0)
    assert bench.capturable(configs.DT, gear.GEAR_OPT_INCREMENTAL_TREE)  # no update in a uniform step
    assert bench.capturable(configs.TINY, 0)                             # one-launch prioritized selection
    assert not bench.capturable(configs.TINY, gear.GEAR_OPT_INCREMENTAL_TREE)
    assert bench.capturable(configs.TOPK_STRESS, 0)
    assert not bench.capturable(configs.MAT, 0)                          # sum tree rebuilt per call
    assert not bench.capturable(configs.GATO_HOST, 0)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "mat", "--graph"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "cannot be replayed" in r.stderr
    assert r.stdout.strip() == ""


def test_group_of_zero_steps_is_refused():
    import pytest
    with pytest.raises(ValueError):
        bench.pipeline_groups(5, 0)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--group", "0"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "--group" in r.stderr


def test_fused_mode_only_for_fifo_lifo_uniform_workloads():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "mat", "--fused"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "--fused" in r.stderr
    assert r.stdout.strip() == ""
