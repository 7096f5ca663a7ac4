"""Typed, named columns at the boundary (Sec. 3.2: fields with names and
per-step shapes fixed at creation; Sec. 3.4: collect(indices, fields)
handed over as tensors).  A MAT-shaped table with bf16 [8, 64]
observations, int32 [8] actions and a float32 reward is filled from typed
tensors keyed by name; the batch from collect_fields is compared with the
oracle's bytes, viewed as the same types and shapes."""
import numpy as np
import pytest
import torch

import gen
import oracle
from paper_2310_05205_amd import gear
from tests.helpers import cuda, host, say

pytestmark = pytest.mark.gpu

COLS = (gen.Column("obs", gen.NORMAL_BF16, 8 * 64, dtype="bf16"),
        gen.Column("action", gen.INT_MOD, 8, param=16, dtype="i32"),
        gen.Column("reward", gen.NORMAL_F32, 1, dtype="f32"))
SPECS = [("obs", torch.bfloat16, (8, 64)), ("action", "int32", (8,)), ("reward", "float32", ())]


def _rows(N, T, seed):
    return [gen.fill_rows_cpu(c, ci, seed, T, 0, N) for ci, c in enumerate(COLS)]


def test_typed_table_collect_fields_matches_oracle():
    N, T, B, L, seed = 3000, 40, 500, 7, 11
    say("typed columns: N=%d T=%d B=%d L=%d" % (N, T, B, L))
    rows = _rows(N, T, seed)
    prio = gen.insert_priorities(gen.PrioDist(gen.PRIO_UNIFORM, 1, 1000), seed, 0, N)
    t = gear.Table(SPECS, N, T)
    try:
        assert [c.name for c in t.columns] == ["obs", "action", "reward"]
        assert [c.elem_bytes for c in t.columns] == [1024, 32, 4]
        assert gear.gear_table_column_info(t.handle, 0) == ("obs", gear.GEAR_DTYPE_BF16, 512)
        assert t.column_index("reward") == 2
        with pytest.raises(gear.GearError):
            t.column_index("done")
        # Typed sources keyed by name, in another order than the columns.
        src = {"reward": torch.from_numpy(rows[2]).view(torch.float32).view(N, T).to(cuda()),
               "obs": torch.from_numpy(rows[0]).view(torch.bfloat16).view(N, T, 8, 64).to(cuda()),
               "action": torch.from_numpy(rows[1]).view(torch.int32).view(N, T, 8).to(cuda())}
        t.insert(src, torch.from_numpy(prio.view(np.int32)).to(cuda()))
        idx, start, w = t.select(gear.GEAR_PRIORITIZED, B, L, seed, 0.4, weights=True)
        batch = t.collect_fields(idx, start, L)
        assert set(batch) == {"obs", "action", "reward"}
        assert batch["obs"].dtype == torch.bfloat16 and tuple(batch["obs"].shape) == (B, L, 8, 64)
        assert batch["action"].dtype == torch.int32 and tuple(batch["action"].shape) == (B, L, 8)
        assert batch["reward"].dtype == torch.float32 and tuple(batch["reward"].shape) == (B, L)

        store = oracle.Store([c.elem_bytes for c in COLS], N, T)
        store.insert(rows, prio)
        st, oidx, ostart, _ = store.select(oracle.PRIORITIZED, B, L, seed, 0.4, weights=True)
        assert st == oracle.OK
        np.testing.assert_array_equal(host(idx), oidx)
        _, ref = store.collect(oidx, ostart, L)
        for (name, dtype, shape), r in zip(SPECS, ref):
            expect = torch.from_numpy(r).view(getattr(torch, str(dtype).replace("torch.", ""))).view((B, L) + shape)
            got = batch[name].cpu()
            assert torch.equal(got.view(torch.uint8), expect.view(torch.uint8)), name
            if name != "obs":
                assert torch.equal(got, expect), name
        # A subset of fields, in a different order, is a subset of the same batch.
        part = t.collect_fields(idx, start, L, fields=["reward", "obs"])
        assert list(part) == ["reward", "obs"]
        assert torch.equal(part["reward"], batch["reward"])
        assert torch.equal(part["obs"].view(torch.uint8), batch["obs"].view(torch.uint8))
        # Uniform selection inside the gather launch hands out the same typed views.
        uidx, ustart, _, ubatch = t.select_collect_fields(gear.GEAR_UNIFORM, B, L, seed + 1, fields=["action", "obs"])
        assert list(ubatch) == ["action", "obs"]
        assert tuple(ubatch["obs"].shape) == (B, L, 8, 64) and ubatch["action"].dtype == torch.int32
        st, oidx, ostart, _ = store.select(oracle.UNIFORM, B, L, seed + 1)
        assert st == oracle.OK
        np.testing.assert_array_equal(host(uidx), oidx)
        np.testing.assert_array_equal(host(ustart), ostart)
        _, ref = store.collect(oidx, ostart, L)
        assert torch.equal(ubatch["action"].cpu().view(torch.uint8).reshape(-1),
                           torch.from_numpy(ref[1]).reshape(-1))
        assert torch.equal(ubatch["obs"].cpu().view(torch.uint8).reshape(-1), torch.from_numpy(ref[0]).reshape(-1))
        assert t.sync() == 0
    finally:
        t.close()


def test_byte_columns_have_default_names():
    t = gear.Table([4, 12], 16, 3)
    try:
        assert [(c.name, c.dtype, c.shape) for c in t.columns] == [("c0", gear.GEAR_DTYPE_U8, (4,)),
                                                                   ("c1", gear.GEAR_DTYPE_U8, (12,))]
        assert t.column_index("c1") == 1
    finally:
        t.close()
