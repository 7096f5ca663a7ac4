"""Selection and updates overlapping the gather on a second stream give the
serial results bit for bit, in the issue order of the benchmark's headline.

Stream S runs the selects and updates of a group of steps and records one
event after the group's last select; stream C waits for it and runs the
group's gathers.  Groups follow the benchmark's schedule (one step, two,
then `group`), the gathers of the first groups run with
GEAR_OPT_GATHER_SHARE_CU as there, and S reuses a buffer set only after C's
event for the group that last used it.  The same table is also driven
serially, on one stream, from the same insertions and seeds.  Indices,
window starts, IS weights, every gathered byte and the final priorities
must agree exactly, so the overlap changes timing only.  Run twice in each
mode, this also checks that the same seeds give the same bytes (no race
decides an output)."""
import numpy as np
import pytest
import torch

import bench
import gen
from gen import configs
from paper_2310_05205_amd import gear
from tests.helpers import cuda, gpu_table, host, say

pytestmark = pytest.mark.gpu

W = configs.Workload(
    name="pipeline N=20000 T=64 B=1024 L=16", seed=41, N=20000, T=64,
    columns=(gen.Column("obs", gen.NORMAL_BF16, 8 * 16, dtype="bf16"),
             gen.Column("action", gen.INT_MOD, 8, param=16, dtype="i32"),
             gen.Column("reward", gen.NORMAL_F32, 1, dtype="f32")),
    n_insert=20000, prio=gen.PrioDist(gen.PRIO_LOGNORMAL, 6.931471805599453, 1.0, float(1 << 24)),
    strategies=(gear.GEAR_PRIORITIZED,), B=1024, L=16, weights=True)
STEPS = 12


def _run(pipelined, group=4):
    t = gpu_table(W)
    dev = cuda()
    nsets = 2 * group if pipelined else 1
    idx = [torch.empty(W.B, dtype=torch.int64, device=dev) for _ in range(nsets)]
    start = [torch.empty(W.B, dtype=torch.int32, device=dev) for _ in range(nsets)]
    wts = [torch.empty(W.B, dtype=torch.float32, device=dev) for _ in range(nsets)]
    outs = [[torch.empty(W.B * W.L * e, dtype=torch.uint8, device=dev) for e in W.elem_bytes] for _ in range(nsets)]
    newp = [torch.from_numpy(gen.update_priorities(W.prio, W.seed, it, W.B).view(np.int32)).to(dev)
            for it in range(STEPS)]
    record = []
    try:
        if not pipelined:
            s = torch.cuda.current_stream(dev).cuda_stream
            for it in range(STEPS):
                gear.gear_select(t.handle, gear.GEAR_PRIORITIZED, W.B, W.L, gen.select_seed(W.seed, it), W.beta,
                                 idx[0].data_ptr(), start[0].data_ptr(), wts[0].data_ptr(), s)
                gear.gear_collect(t.handle, idx[0].data_ptr(), start[0].data_ptr(), W.B, W.L, None,
                                  [o.data_ptr() for o in outs[0]], s)
                gear.gear_update_priorities(t.handle, idx[0].data_ptr(), newp[it].data_ptr(), W.B, s)
                record.append([host(idx[0]), host(start[0]), host(wts[0])] + [host(o) for o in outs[0]])
        else:
            C, S = torch.cuda.Stream(dev), torch.cuda.Stream(dev)
            groups = bench.pipeline_groups(STEPS, group)
            sel_done = [torch.cuda.Event() for _ in groups]
            col_done = [torch.cuda.Event() for _ in groups]
            pending = []  # gathered steps not yet read back, in step order

            def read_back():
                torch.cuda.synchronize(dev)
                for j in pending:
                    k = j % nsets
                    record.append([host(idx[k]), host(start[k]), host(wts[k])] + [host(o) for o in outs[k]])
                pending.clear()

            for g, (js, waits) in enumerate(zip(groups, bench.set_reuse_waits(groups, nsets))):
                if {j % nsets for j in js} & {j % nsets for j in pending}:
                    read_back()  # before the group rewrites a set
                for p in waits:
                    S.wait_event(col_done[p])
                for n, j in enumerate(js):
                    k = j % nsets
                    gear.gear_select(t.handle, gear.GEAR_PRIORITIZED, W.B, W.L, gen.select_seed(W.seed, j), W.beta,
                                     idx[k].data_ptr(), start[k].data_ptr(), wts[k].data_ptr(), S.cuda_stream)
                    if n == len(js) - 1:
                        sel_done[g].record(S)
                    gear.gear_update_priorities(t.handle, idx[k].data_ptr(), newp[j].data_ptr(), W.B, S.cuda_stream)
                C.wait_event(sel_done[g])
                t.set_options(gear.GEAR_OPT_GATHER_SHARE_CU if g < len(bench.RAMP) else 0)
                for j in js:
                    k = j % nsets
                    gear.gear_collect(t.handle, idx[k].data_ptr(), start[k].data_ptr(), W.B, W.L, None,
                                      [o.data_ptr() for o in outs[k]], C.cuda_stream)
                col_done[g].record(C)
                pending.extend(js)
            t.set_options(0)
            read_back()
        torch.cuda.synchronize(dev)
        assert t.sync() == 0
        return record, t.priorities()
    finally:
        t.close()


def test_pipelined_issue_order_matches_serial_bit_for_bit():
    say("pipeline: serial reference")
    ref, ref_p = _run(False)
    for group in (2, 4):
        say("pipeline: two streams, %d steps per handshake" % group)
        got, got_p = _run(True, group)
        assert len(got) == len(ref) == STEPS
        for it, (a, b) in enumerate(zip(ref, got)):
            for x, y in zip(a, b):
                np.testing.assert_array_equal(x, y, err_msg="step %d" % it)
        np.testing.assert_array_equal(ref_p, got_p)
    say("pipeline: serial again")
    again, again_p = _run(False)
    for a, b in zip(ref, again):
        for x, y in zip(a, b):
            np.testing.assert_array_equal(x, y)
    np.testing.assert_array_equal(ref_p, again_p)
