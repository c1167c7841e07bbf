"""dpi_lookup_noalloc (plan and lookup with the library's fixed device scratch)
against dpi_plan + dpi_lookup with a caller workspace, through the C ABI:
bit for bit on two calls in a row, the second with a smaller batch, plus the
error paths (a batch too large for the scratch, an id outside its table)."""
import numpy as np
import pytest
import torch

from paper_2606_21101_amd import dpi
from paper_2606_21101_amd.lookup import FusedLookup
from parity import gpu_tables, out_torch_dtype, pooling_codes
from synth import configs, generate as G

pytestmark = pytest.mark.gpu


def _both(cfg, tables, batch):
    out_dt = out_torch_dtype(cfg)
    pool = pooling_codes(cfg)
    fl = FusedLookup(tables, pool, out_dt, num_rows=G.table_sizes(cfg))
    ref = fl(batch.ids, batch.offsets, cfg.batch)
    out = torch.full_like(ref, float("nan"))
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    print(f"  noalloc: config {cfg.key} B={cfg.batch}", flush=True)
    dpi.dpi_lookup_noalloc(fl.meta, tables, batch.ids, batch.offsets, cfg.batch, batch.total_ids, pool,
                           fl.opts(), out, status)
    torch.cuda.synchronize()
    return ref, out, int(status.item())


def test_noalloc_matches_workspace_path_twice():
    """The multi-hot workload (the plan's partition), then the heterogeneous sweep
    at B = 128 (a smaller batch, bag by bag): same output bits as the caller-
    workspace path, status 0."""
    cfg = configs.get(3)
    tables = gpu_tables(cfg)
    batch = G.make_batch(cfg, device="cuda")
    ref, out, st = _both(cfg, tables, batch)
    assert st == 0
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    del tables, batch
    cfg2 = configs.get(5, batch=128)
    tables2 = gpu_tables(cfg2)
    batch2 = G.make_batch(cfg2, device="cuda")
    ref2, out2, st2 = _both(cfg2, tables2, batch2)
    assert st2 == 0
    assert torch.equal(out2.view(torch.int32), ref2.view(torch.int32))


def test_noalloc_one_hot_and_bad_id():
    """A one-hot batch (no offsets) equal to the workspace path, then the same
    batch with one id outside its table: reported in the device status word."""
    cfg = configs.get(2)
    tables = gpu_tables(cfg)
    batch = G.make_batch(cfg, device="cuda")
    ref, out, st = _both(cfg, tables, batch)
    assert st == 0
    assert torch.equal(out.view(torch.int32), ref.view(torch.int32))
    bad_ids = batch.ids.clone()
    bad_ids[5] = int(G.table_sizes(cfg)[0])              # one past field 0's last row
    fl = FusedLookup(tables, None, torch.float32, num_rows=G.table_sizes(cfg))
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    dpi.dpi_lookup_noalloc(fl.meta, tables, bad_ids, None, cfg.batch, batch.total_ids, None, fl.opts(),
                           torch.empty_like(ref), status)
    torch.cuda.synchronize()
    assert int(status.item()) == dpi.DPI_DEVSTAT_BAD_ID


def test_noalloc_rejects_a_batch_beyond_the_scratch():
    """A wave count whose per-wave state exceeds the fixed scratch is refused
    before anything is enqueued."""
    tabs = [torch.zeros((10, 16), device="cuda")]
    fl = FusedLookup(tabs)
    B = 1 << 20
    ids = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.full((B, 16), 3.0, device="cuda")
    with pytest.raises(dpi.DpiError) as e:
        dpi.dpi_lookup_noalloc(fl.meta, tabs, ids, None, B, B, None, fl.opts(num_waves=B), out)
    assert e.value.status == dpi.DPI_ERR_WORKSPACE_TOO_SMALL
    assert "scratch" in dpi.dpi_last_error()
    torch.cuda.synchronize()
    assert torch.all(out == 3.0)


def test_noalloc_long_bags_and_bad_offsets():
    """A small batch with long bags (one launch per lookup: the long bags pooled
    in pieces over their fields' waves) bit for bit against the workspace path,
    then malformed offsets reported in the device status word."""
    from test_gpu_edges import random_problem
    rng = np.random.default_rng(31)
    B = 40
    tables, _, offs0, pool = random_problem(rng, [16, 64], [0, 1], B, 10, rows=300)
    lens = np.diff(offs0, axis=1).astype(np.int64)
    lens[1, 5] = 3000
    lens[0, 39] = 200
    offs = np.zeros((2, B + 1), np.int32)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    ids = np.concatenate([rng.integers(0, 300, int(offs[t, -1])) for t in range(2)]).astype(np.int32)
    tt = [torch.from_numpy(t).cuda() for t in tables]
    ids_d, offs_d = torch.from_numpy(ids).cuda(), torch.from_numpy(offs).cuda()
    fl = FusedLookup(tt, pool)
    ref = fl(ids_d, offs_d, B)
    out = torch.full_like(ref, float("nan"))
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    print(f"  noalloc: long bags B={B}", flush=True)
    dpi.dpi_lookup_noalloc(fl.meta, tt, ids_d, offs_d, B, len(ids), pool, fl.opts(), out, status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert torch.equal(out.view(torch.int32), ref.view(torch.int32))
    bad = offs.copy()
    bad[0, 3] = bad[0, 2] - 1
    status.fill_(-1)
    dpi.dpi_lookup_noalloc(fl.meta, tt, ids_d, torch.from_numpy(bad).cuda(), B, len(ids), pool, fl.opts(),
                           torch.empty_like(ref), status)
    torch.cuda.synchronize()
    assert int(status.item()) == dpi.DPI_DEVSTAT_BAD_OFFSETS
