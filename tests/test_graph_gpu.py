"""HIP graph capture of gear_collect, the one hot-path call that keeps no
host-side state.  A captured collect is replayed several times; between
replays new draws are written into its index and start buffers by eager
work, and every replay must equal the oracle's windows for those draws.
"""
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
