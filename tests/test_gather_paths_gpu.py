"""The gather moves 8 elements per thread for batches of at least 128 MiB
and 2 for smaller ones.  A batch just above that size and the same windows
minus the last one, just below it, are gathered from one HBM table and
compared byte for byte with each other and with plain torch indexing of the
table's columns (Sec. 3.4 collection: batch row b is the window of slot
idx[b] that starts at step start[b])."""
import pytest
import torch

from paper_2310_05205_amd import gear
from tests.helpers import cuda, say

pytestmark = pytest.mark.gpu

LARGE = 128 << 20


def _reference(t, idx, start, L):
    outs = []
    for c, e in enumerate(t.elem_bytes):
        col = t.column_view(c).view(t.capacity, t.T, e)
        steps = start.long()[:, None] + torch.arange(L, device=idx.device)[None, :]
        outs.append(col[idx[:, None], steps].reshape(idx.shape[0], L * e))
    return outs


# L = T: whole trajectories, moved with the trajectory as the source stride;
# L < T: windows inside them.  The 4-byte column is narrow on both sides.
@pytest.mark.parametrize("L", [64, 48])
def test_both_sides_of_the_large_batch_size(L):
    N, T, eb = 4096, 64, [1024, 4]
    per_window = L * sum(eb)
    big = -(-LARGE // per_window)
    small = big - 1
    assert small * per_window < LARGE <= big * per_window
    say("gather paths: L=%d, %d windows (%d bytes) and %d (%d bytes)"
        % (L, big, big * per_window, small, small * per_window))
    g = torch.Generator(device=cuda()).manual_seed(5)
    t = gear.Table(eb, N, T, gear.GEAR_DEVICE, 0)
    try:
        rows = [torch.randint(0, 256, (N, T * e), dtype=torch.uint8, device=cuda(), generator=g) for e in eb]
        t.insert(rows, torch.ones(N, dtype=torch.int32, device=cuda()))
        idx, start, _ = t.select(gear.GEAR_UNIFORM, big, L, 77)
        out_big = t.collect(idx, start, L)
        out_small = t.collect(idx[:small], start[:small], L)
        ref = _reference(t, idx, start, L)
        torch.cuda.synchronize()
        for c in range(len(eb)):
            assert torch.equal(out_big[c], ref[c]), "column %d, %d windows" % (c, big)
            assert torch.equal(out_small[c], ref[c][:small]), "column %d, %d windows" % (c, small)
        assert t.sync() == 0
    finally:
        t.close()


# 4096 whole 64-step windows of 1 KiB steps make 8192 workgroups of the
# 1 KiB column, enough for a gather that caps its workgroups per CU.
# GEAR_OPT_GATHER_SHARE_CU only lowers that cap: the bytes are the same.
def test_share_option_moves_the_same_bytes():
    N, T, L, eb = 4096, 64, 64, [1024, 4]
    g = torch.Generator(device=cuda()).manual_seed(9)
    t = gear.Table(eb, N, T, gear.GEAR_DEVICE, 0)
    try:
        rows = [torch.randint(0, 256, (N, T * e), dtype=torch.uint8, device=cuda(), generator=g) for e in eb]
        t.insert(rows, torch.ones(N, dtype=torch.int32, device=cuda()))
        idx, start, _ = t.select(gear.GEAR_UNIFORM, N, L, 78)
        say("share option: %d windows of %d bytes" % (N, L * sum(eb)))
        plain = t.collect(idx, start, L)
        t.set_options(gear.GEAR_OPT_GATHER_SHARE_CU)
        shared = t.collect(idx, start, L)
        t.set_options(0)
        again = t.collect(idx, start, L)
        ref = _reference(t, idx, start, L)
        torch.cuda.synchronize()
        for c in range(len(eb)):
            assert torch.equal(plain[c], ref[c]), "column %d" % c
            assert torch.equal(shared[c], ref[c]), "column %d, shared" % c
            assert torch.equal(again[c], ref[c]), "column %d, option off again" % c
        with pytest.raises(gear.GearError):
            t.set_options(8)
        assert t.sync() == 0
    finally:
        t.close()
