"""Seeded random problems across every lookup path (partition, bag by bag,
one-hot, input-first, long-bag fallback), each checked against the oracle,
and the exported plan against the plan oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_21101_amd import dpi
from paper_2606_21101_amd.lookup import FusedLookup
from test_gpu_edges import check

pytestmark = pytest.mark.gpu
PLAN_KEYS = ("header", "col_base", "id_base", "bag_item_base", "bag_cost_base", "wave_item_begin")


def random_case(seed):
    rng = np.random.default_rng(9000 + seed)
    T = int(rng.integers(1, 13))
    fast = rng.random() < 0.7                     # every row a multiple of 16 bytes (bag-by-bag eligible)
    dims, dtypes = [], []
    for _ in range(T):
        dt = int(rng.integers(0, 2))
        if fast:
            d = int(rng.choice([8, 16, 32, 64, 128, 256, 512])) // (1 + dt) * (1 + dt)
            d = d if dt else d // 2 * 2
            d = max(d, 4 if dt == 0 else 8)
        else:
            d = int(rng.integers(1, 300)) * (2 if dt else 1)
        dims.append(d)
        dtypes.append(dt)
    B = int(rng.choice([0, 1, 2, 7, 33, 100, 257, 600]))
    rows = [int(rng.integers(1, 400)) for _ in range(T)]
    mode = rng.integers(0, 4)
    if mode == 0:
        lens = np.ones((T, B), np.int64)                        # one-hot through offsets
    elif mode == 1:
        lens = rng.poisson(rng.uniform(0.5, 12), size=(T, B))  # short bags, some empty
    elif mode == 2:
        lens = rng.integers(0, 40, size=(T, B))
        if B:
            lens[int(rng.integers(0, T)), int(rng.integers(0, B))] = int(rng.integers(129, 900))   # a long bag
    else:
        lens = np.minimum(np.floor(rng.lognormal(np.log(6), 1.0, size=(T, B))), 300).astype(np.int64)
    offs = np.zeros((T, B + 1), np.int32)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    ids = np.concatenate([rng.integers(0, rows[t], int(offs[t, -1])) for t in range(T)] + [np.zeros(0)]).astype(np.int32)
    tables = [(rng.standard_normal((rows[t], dims[t])) * 0.01).astype(np.float16 if dtypes[t] else np.float32)
              for t in range(T)]
    pool = [int(x) for x in rng.integers(0, 2, T)]
    flags = int(rng.choice([0, 0, 0, dpi.DPI_FLAG_EXACT_SPLIT, dpi.DPI_FLAG_LINEAR_BLOCKS, dpi.DPI_FLAG_INPUT_FIRST]))
    waves = int(rng.choice([0, 0, 1, 3, 50, 1000]))
    chunk = int(rng.choice([0, 0, 1, 8]))
    out_dtype = torch.float16 if rng.random() < 0.4 else torch.float32
    null_offsets = mode == 0 and rng.random() < 0.5
    return dims, dtypes, tables, ids, (None if null_offsets else offs), pool, B, flags, waves, chunk, out_dtype


@pytest.mark.parametrize("seed", range(48))
def test_fuzz(seed):
    dims, dtypes, tables, ids, offs, pool, B, flags, waves, chunk, od = random_case(seed)
    tt = [torch.from_numpy(t).cuda() for t in tables]
    fl = FusedLookup(tt, pool, od, chunk_rows=chunk, flags=flags)
    ids_d = torch.from_numpy(ids).cuda()
    offs_d = None if offs is None else torch.from_numpy(offs).cuda()
    plan = fl.plan(offs_d, B, len(ids), num_waves=waves)
    out = fl.lookup(plan, ids_d, offs_d)
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_OK
    onehot = offs is None or (len(ids) == len(dims) * B and np.all(np.diff(offs, axis=1) == 1))
    check(tables, ids, offs, pool, B, out, exact=onehot and od == torch.float32)
    got = dpi.dpi_plan_export(plan)
    W = waves if waves else dpi.dpi_default_waves(len(dims), B, len(ids))
    ref = oracle.plan(dims, dtypes, 1 if od == torch.float16 else 0, offs, B, len(ids), chunk or 32, 64, W, flags)
    for k in PLAN_KEYS:
        assert np.array_equal(got[k], ref[k]), (seed, k)
    out2 = fl.lookup(plan, ids_d, offs_d)       # after the export's full re-plan
    assert torch.equal(out, out2)
