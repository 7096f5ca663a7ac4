"""Separate tables are independent: two tables driven on two HIP streams,
their calls interleaved on the host with no synchronisation between them,
give exactly the oracle's results for each table, iteration by iteration.
"""
import dataclasses

import numpy as np
import pytest
import torch

import gen
import oracle
from gen import configs
from paper_2310_05205_amd import gear
from tests.helpers import assert_weights, cuda, gpu_table, host, oracle_store, say

pytestmark = pytest.mark.gpu


def test_two_tables_on_two_streams():
    ws = [configs.TINY, dataclasses.replace(configs.TINY, seed=11, name="tiny-prioritized seed 11")]
    stores = [oracle_store(w) for w in ws]
    tables = [gpu_table(w) for w in ws]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]   # default priority
    iters = 4
    try:
        torch.cuda.synchronize()
        results = [[None] * iters for _ in ws]
        newps = [[gen.update_priorities(w.prio, w.seed, it, w.B) for it in range(iters)] for w in ws]
        dev_newps = [[torch.from_numpy(p).to(cuda()) for p in ps] for ps in newps]
        torch.cuda.synchronize()
        say("two tables on two streams: %d interleaved iterations" % iters)
        for it in range(iters):
            for k, (w, t, s) in enumerate(zip(ws, tables, streams)):
                with torch.cuda.stream(s):
                    idx, start, wt = t.select(gear.GEAR_PRIORITIZED, w.B, w.L, gen.select_seed(w.seed, it), w.beta,
                                              weights=True)
                    outs = t.collect(idx, start, w.L)
                    t.update_priorities(idx, dev_newps[k][it])
                    results[k][it] = (idx, start, wt, outs)
        torch.cuda.synchronize()
        for k, (w, s_, t) in enumerate(zip(ws, stores, tables)):
            for it in range(iters):
                idx, start, wt, outs = results[k][it]
                st, oidx, ostart, ow = s_.select(gear.GEAR_PRIORITIZED, w.B, w.L, gen.select_seed(w.seed, it), w.beta,
                                                 weights=True)
                assert st == oracle.OK
                np.testing.assert_array_equal(host(idx), oidx)
                np.testing.assert_array_equal(host(start), ostart)
                assert_weights(host(wt), ow)
                st, oouts = s_.collect(oidx, ostart, w.L)
                for c in range(len(w.columns)):
                    np.testing.assert_array_equal(host(outs[c]), oouts[c])
                assert s_.update(oidx, newps[k][it]) == oracle.OK
            np.testing.assert_array_equal(t.priorities(), s_.priority)
            assert t.sync() == 0
    finally:
        for t in tables:
            t.close()
