"""HIP graph capture of the hot-path calls whose captures replay correctly.

A captured collect is replayed several times; between replays new draws are
written into its index and start buffers by eager work, and every replay
must equal the oracle's windows for those draws.

Whole steps (select, collect and, for prioritized and TopK selection, the
priority update; or one gear_select_collect call) of the strategies whose
selection keeps no decision on the host are captured from one table and replayed several times, while a twin
table runs the same steps eagerly; every replay must give the eager run's
indices, starts, weights, batches and priorities bit for bit.
"""
import dataclasses

import numpy as np
import pytest
import torch

import gen
from gen import configs
from paper_2310_05205_amd import gear
from tests.helpers import cuda, gpu_table, host, oracle_priorities, oracle_windows, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("pinned", [False, True], ids=["hbm", "pinned-host"])
def test_captured_collect_replays_new_draws(pinned):
    w = configs.TINY
    _, next_seq = oracle_priorities(w)
    t = gpu_table(w, gear.GEAR_HOST_PINNED if pinned else gear.GEAR_DEVICE)
    try:
        B, L = w.B, 16
        idx = torch.zeros(B, dtype=torch.int64, device=cuda())
        start = torch.zeros(B, dtype=torch.int32, device=cuda())
        outs = [torch.empty((B, L * e), dtype=torch.uint8, device=cuda()) for e in w.elem_bytes]
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            t.collect(idx, start, L, out=outs)
        rng = np.random.default_rng(5)
        for r in range(4):
            say("graph replay %d (%s)" % (r, "pinned" if pinned else "hbm"))
            i = rng.integers(0, w.N, B).astype(np.int64)
            s = rng.integers(0, w.T - L + 1, B).astype(np.int32)
            idx.copy_(torch.from_numpy(i))
            start.copy_(torch.from_numpy(s))
            g.replay()
            torch.cuda.synchronize()
            want = oracle_windows(w, i, s, L, next_seq, np.arange(B))
            for c, o in enumerate(outs):
                np.testing.assert_array_equal(host(o), want[c].reshape(B, -1))
            assert t.sync() == 0
            # eager work between replays, on the same table
            t.select(gear.GEAR_PRIORITIZED, B, L, gen.select_seed(w.seed, r))
            torch.cuda.synchronize()
    finally:
        t.close()


# The DT shape on a small table whose ring has wrapped; the tiny prioritized
# table (4096 slots: selection in one launch, no sum tree).
DT_SMALL = dataclasses.replace(configs.DT, name="dt-small N=4096 T=100 B=512 L=20", N=4096, T=100,
                               n_insert=4096 + 512)
STEP_CASES = [(DT_SMALL, gear.GEAR_UNIFORM, False), (DT_SMALL, gear.GEAR_FIFO, False),
              (DT_SMALL, gear.GEAR_LIFO, False), (configs.TINY, gear.GEAR_PRIORITIZED, False),
              (configs.TINY, gear.GEAR_TOPK, False),
              # one gear_select_collect launch per step
              (DT_SMALL, gear.GEAR_UNIFORM, True), (DT_SMALL, gear.GEAR_FIFO, True), (DT_SMALL, gear.GEAR_LIFO, True)]
STEPS, REPLAYS = 5, 3


def _buffers(w):
    dev = cuda()
    return [(torch.empty(w.B, dtype=torch.int64, device=dev), torch.empty(w.B, dtype=torch.int32, device=dev),
             torch.empty(w.B, dtype=torch.float32, device=dev),
             [torch.empty(w.B * w.L * e, dtype=torch.uint8, device=dev) for e in w.elem_bytes])
            for _ in range(STEPS)]


def _steps(t, w, strategy, bufs, newp, stream, fused=False):
    weights = strategy in (gear.GEAR_PRIORITIZED, gear.GEAR_TOPK)
    for j, (idx, start, wts, outs) in enumerate(bufs):
        if fused:
            gear.gear_select_collect(t.handle, strategy, w.B, w.L, gen.select_seed(w.seed, j), idx.data_ptr(),
                                     start.data_ptr(), wts.data_ptr(), None, [o.data_ptr() for o in outs], stream)
            continue
        gear.gear_select(t.handle, strategy, w.B, w.L, gen.select_seed(w.seed, j), w.beta, idx.data_ptr(),
                         start.data_ptr(), wts.data_ptr() if weights else None, stream)
        gear.gear_collect(t.handle, idx.data_ptr(), start.data_ptr(), w.B, w.L, None, [o.data_ptr() for o in outs],
                          stream)
        if weights:
            gear.gear_update_priorities(t.handle, idx.data_ptr(), newp[j].data_ptr(), w.B, stream)


@pytest.mark.parametrize("w,strategy,fused", STEP_CASES,
                         ids=["dt-uniform", "dt-fifo", "dt-lifo", "tiny-prioritized", "tiny-topk", "dt-uniform-fused",
                              "dt-fifo-fused", "dt-lifo-fused"])
def test_captured_steps_replay_like_eager_steps(w, strategy, fused):
    dev = cuda()
    eager_t, graph_t = gpu_table(w), gpu_table(w)
    try:
        newp = [torch.from_numpy(gen.update_priorities(w.prio, w.seed, j, w.B).view(np.int32)).to(dev)
                for j in range(STEPS)]
        eager_b, graph_b = _buffers(w), _buffers(w)
        side = torch.cuda.Stream(dev)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side, capture_error_mode="relaxed"):
            _steps(graph_t, w, strategy, graph_b, newp, side.cuda_stream, fused)
        scratch = [torch.empty(w.B * w.L * e, dtype=torch.uint8, device=dev) for e in w.elem_bytes]
        for r in range(REPLAYS):
            say("captured steps: %s strategy %d, replay %d" % (w.name, strategy, r))
            _steps(eager_t, w, strategy, eager_b, newp, torch.cuda.current_stream(dev).cuda_stream, fused)
            g.replay()
            torch.cuda.synchronize()
            nout = 3 if fused or strategy in (gear.GEAR_PRIORITIZED, gear.GEAR_TOPK) else 2  # weights written or not
            for j, (a, b) in enumerate(zip(eager_b, graph_b)):
                for x, y in zip(a[:nout], b[:nout]):
                    np.testing.assert_array_equal(host(x), host(y), err_msg="replay %d step %d" % (r, j))
                for x, y in zip(a[3], b[3]):
                    assert torch.equal(x, y), "replay %d step %d" % (r, j)
            np.testing.assert_array_equal(eager_t.priorities(), graph_t.priorities(), err_msg="replay %d" % r)
            # eager work on the captured table between replays: a gather that only reads it
            idx, start = graph_b[0][0], graph_b[0][1]
            gear.gear_collect(graph_t.handle, idx.data_ptr(), start.data_ptr(), w.B, w.L, None,
                              [o.data_ptr() for o in scratch], torch.cuda.current_stream(dev).cuda_stream)
            torch.cuda.synchronize()
            for x, y in zip(scratch, graph_b[0][3]):
                assert torch.equal(x, y)
        assert eager_t.sync() == 0 and graph_t.sync() == 0
    finally:
        eager_t.close()
        graph_t.close()
