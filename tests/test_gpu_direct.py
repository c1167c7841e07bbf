"""Small batches looked up bag by bag (no partition), against the oracle.

With the wave count left to the library, a batch of at most 180,000 bags whose
fields all take the 16-byte row path is pooled bag by bag.  Up to 64 fields
and 1024 bags per field that is one launch per lookup, which pools a bag of
more than four chunks in pieces over the field's waves; larger batches are
planned by their own launch first, and a bag of more than four chunks anywhere
in the batch sends the lookup to the plan's partition.  Every case is also run
with an explicit wave count (the plan's partition) and both results are
checked against the oracle.
"""
import numpy as np
import pytest
import torch

from paper_2606_21101_amd import dpi
from test_gpu_edges import check, random_problem, run_case

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("B", [1, 2, 3, 5, 33, 100, 257])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.float16])
def test_direct_mixed_classes(B, out_dtype):
    # rows of 16 .. 1024 bytes: 64 down to 1 slots per wave, fp16 and fp32
    dims = [4, 8, 16, 32, 64, 128, 256, 8, 64, 512]
    dtypes = [0, 0, 0, 0, 0, 0, 0, 1, 1, 1]
    rng = np.random.default_rng(1000 + B)
    tables, ids, offs, pool = random_problem(rng, dims, dtypes, B, 40, rows=300)
    out, st, _, _ = run_case(tables, ids, offs, pool, B, out_dtype)
    assert st == dpi.DPI_OK
    check(tables, ids, offs, pool, B, out)
    out_p, st_p, _, _ = run_case(tables, ids, offs, pool, B, out_dtype, num_waves=7)
    assert st_p == dpi.DPI_OK
    check(tables, ids, offs, pool, B, out_p)


@pytest.mark.parametrize("B", [1, 4, 64])
def test_direct_one_field_long_bags_up_to_the_limit(B):
    # bags of up to 4 chunks of 32 ids (128 rows) stay on the bag-by-bag path
    rng = np.random.default_rng(7 + B)
    tables, ids, offs, pool = random_problem(rng, [32], [1], B, 128, rows=1000, p_empty=0.2)
    offs[0, 1:] = np.cumsum(np.r_[128, np.diff(offs[0])[1:]])   # the first bag has exactly 128 ids
    ids = rng.integers(0, 1000, int(offs[0, -1])).astype(np.int32)
    for pool_t in ([0], [1]):
        out, st, _, _ = run_case(tables, ids, offs, pool_t, B)
        assert st == dpi.DPI_OK
        check(tables, ids, offs, pool_t, B, out)


@pytest.mark.parametrize("long_len", [129, 1000, 20000])
def test_direct_long_bag(long_len):
    rng = np.random.default_rng(long_len)
    B = 20
    tables, ids, offs, pool = random_problem(rng, [16, 64, 8], [0, 1, 0], B, 30, rows=500)
    lens = np.diff(offs, axis=1)
    lens[1, 7] = long_len
    offs[:, 1:] = np.cumsum(lens, axis=1)
    ids = np.concatenate([rng.integers(0, 500, int(offs[t, -1])) for t in range(3)]).astype(np.int32)
    for od in (torch.float32, torch.float16):
        out, st, _, _ = run_case(tables, ids, offs, pool, B, od)
        assert st == dpi.DPI_OK
        check(tables, ids, offs, pool, B, out)


def test_direct_onehot_mixed_classes_bit_exact():
    # NULL offsets with fields of different row classes take the bag-by-bag path
    rng = np.random.default_rng(11)
    dims, dtypes, B = [16, 8, 64, 4], [0, 1, 1, 0], 77
    tables, _, _, pool = random_problem(rng, dims, dtypes, B, 1, rows=90)
    ids = np.concatenate([rng.integers(0, 90, B) for _ in dims]).astype(np.int32)
    for od in (torch.float32, torch.float16):
        out, st, _, _ = run_case(tables, ids, None, pool, B, od)
        assert st == dpi.DPI_OK
        if od == torch.float32:
            check(tables, ids, None, pool, B, out, exact=True)
        else:
            check(tables, ids, None, pool, B, out)


def test_direct_empty_bags_and_signed_zero():
    rng = np.random.default_rng(12)
    tables, _, _, _ = random_problem(rng, [16, 32], [0, 1], 9, 3, rows=20)
    tables[0][3] = -0.0
    offs = np.array([[0, 0, 1, 1, 3, 3, 3, 4, 4, 4], [0, 0, 0, 0, 0, 0, 0, 0, 0, 2]], np.int32)
    ids = np.array([3, 3, 3, 5, 1, 2], np.int32)
    out, st, _, _ = run_case(tables, ids, offs, [0, 1], 9)
    assert st == dpi.DPI_OK
    check(tables, ids, offs, [0, 1], 9, out)
    y = out.cpu().numpy()
    assert np.all(y[[0, 2, 4, 5, 7, 8], :16] == 0)
    assert not np.signbit(y[1, :16]).any()          # a pooled -0 row is +0, as on every path
    assert np.all(y[:8, 16:] == 0)


def test_direct_bad_ids_reported_and_skipped():
    rng = np.random.default_rng(13)
    tables, ids, offs, pool = random_problem(rng, [16, 8], [0, 0], 12, 6, p_empty=0.0)
    bad_ids = ids.copy()
    bad_ids[2] = -5
    bad_ids[len(ids) - 1] = 50
    out, st, _, _ = run_case(tables, bad_ids, offs, [0, 0], 12)
    assert st == dpi.DPI_ERR_BAD_ID
    fixed = bad_ids.copy()
    fixed[fixed < 0] = 50
    tables_z = [np.concatenate([t, np.zeros((1, t.shape[1]), t.dtype)]) for t in tables]
    check(tables_z, fixed, offs, [0, 0], 12, out)


@pytest.mark.parametrize("B", [2, 2000])
def test_direct_bad_offsets_reported_and_their_field_not_written(B):
    # one launch (B = 2) and planned by its own launch (B = 2000)
    tabs = [torch.zeros((10, 16), device="cuda"), torch.zeros((10, 8), device="cuda", dtype=torch.float16)]
    from paper_2606_21101_amd.lookup import FusedLookup
    fl = FusedLookup(tabs)
    offs_np = np.stack([np.arange(B + 1), np.arange(B + 1)]).astype(np.int32)
    offs_np[0, 1] = 2
    offs_np[0, 2] = 1                      # field 0 decreases
    offs = torch.from_numpy(offs_np).cuda()
    total = int(offs_np[:, -1].sum())
    plan = fl.plan(offs, B, total)
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_ERR_BAD_OFFSETS
    out = torch.full((B, 24), 7.0, device="cuda")
    fl.lookup(plan, torch.zeros(total, dtype=torch.int32, device="cuda"), offs, out)
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_ERR_BAD_OFFSETS
    assert torch.all(out[:, :16] == 7.0)


def test_direct_repeated_lookups_deterministic():
    rng = np.random.default_rng(14)
    tables, ids, offs, pool = random_problem(rng, [64, 16, 8], [1, 0, 0], 50, 60)
    a, _, _, _ = run_case(tables, ids, offs, pool, 50)
    b, _, _, _ = run_case(tables, ids, offs, pool, 50)
    assert torch.equal(a, b)


# --- the plan of a bag-by-bag batch: partition computed on export -----------

import oracle                                   # noqa: E402
from parity import check_outputs, default_waves, oracle_ref, plan_args   # noqa: E402
from synth import configs, generate as G        # noqa: E402
from paper_2606_21101_amd.lookup import FusedLookup   # noqa: E402

PLAN_KEYS = ("header", "col_base", "id_base", "bag_item_base", "bag_cost_base", "wave_item_begin")


def assert_plan_equals_oracle(got, dims, dtypes, out_dtype, offs_np, B, total, W):
    ref = oracle.plan(dims, dtypes, out_dtype, offs_np, B, total, 32, 64, W, 0)
    for k in PLAN_KEYS:
        assert np.array_equal(got[k], ref[k]), (k, got[k][:20], ref[k][:20])


@pytest.mark.parametrize("batch", [1, 16, 128, 512])
def test_lazy_partition_export_matches_oracle(batch):
    cfg = configs.get(5, batch=batch)
    tables = [G.make_table(cfg, t, "cuda") for t in range(cfg.num_tables)]
    b = G.make_batch(cfg, device="cuda")
    dims, dtypes, out_dtype = plan_args(cfg)
    fl = FusedLookup(tables, None, torch.float32, num_rows=G.table_sizes(cfg))
    offs_np = b.offsets.cpu().numpy()
    total = int(b.total_ids)
    W = default_waves(cfg, total)
    # lookup first (no partition computed), then export, then a second lookup
    plan = fl.plan(b.offsets, cfg.batch, total)
    out1 = fl.lookup(plan, b.ids, b.offsets)
    got = dpi.dpi_plan_export(plan)
    assert_plan_equals_oracle(got, dims, dtypes, out_dtype, offs_np, cfg.batch, total, W)
    out2 = fl.lookup(plan, b.ids, b.offsets)
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_OK
    assert torch.equal(out1, out2)
    # export straight after planning
    plan2 = fl.plan(b.offsets, cfg.batch, total)
    got2 = dpi.dpi_plan_export(plan2)
    assert_plan_equals_oracle(got2, dims, dtypes, out_dtype, offs_np, cfg.batch, total, W)
    assert torch.equal(fl.lookup(plan2, b.ids, b.offsets), out1)
    p, ref, mag = oracle_ref(cfg)
    y = out1[torch.from_numpy(p["samples"]).cuda()].double().cpu().numpy()
    check_outputs(y, ref, mag, False, False)


def test_lazy_partition_long_bag_export_matches_oracle():
    rng = np.random.default_rng(21)
    B, dims, dtypes = 30, [16, 64], [0, 1]
    lengths = rng.integers(0, 20, size=(2, B))
    lengths[0, 3] = 300                                  # more than 4 items: partition in the planning launch
    offs_np = G.offsets_from_lengths(lengths)
    total = int(lengths.sum())
    tabs = [torch.zeros((5, d), dtype=torch.float16 if dt else torch.float32, device="cuda")
            for d, dt in zip(dims, dtypes)]
    fl = FusedLookup(tabs)
    plan = fl.plan(torch.from_numpy(offs_np).cuda(), B, total)
    got = dpi.dpi_plan_export(plan)
    W = dpi.dpi_default_waves(2, B, total)
    assert_plan_equals_oracle(got, dims, dtypes, 0, offs_np, B, total, W)


def test_lazy_partition_export_keeps_bad_id_status():
    rng = np.random.default_rng(22)
    tables, ids, offs, pool = random_problem(rng, [16, 8], [0, 0], 12, 6, p_empty=0.0)
    ids = ids.copy()
    ids[1] = 77                                          # outside the 50-row table
    out, st, fl, plan = run_case(tables, ids, offs, pool, 12)
    assert st == dpi.DPI_ERR_BAD_ID
    dpi.dpi_plan_export(plan)                            # plans again with the partition
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_ERR_BAD_ID


@pytest.mark.parametrize("B", [45000, 45001])
def test_bag_limit_both_sides(B):
    # 4 fields: 180000 bags (bag by bag) and 180004 bags (the partition), short bags
    rng = np.random.default_rng(B)
    dims, dtypes = [16, 8, 32, 64], [0, 1, 0, 1]
    tables, ids, offs, pool = random_problem(rng, dims, dtypes, B, 6, rows=2000)
    for od in (torch.float32, torch.float16):
        out, st, _, plan = run_case(tables, ids, offs, pool, B, od)
        assert st == dpi.DPI_OK
        check(tables, ids, offs, pool, B, out)
    got = dpi.dpi_plan_export(plan)
    W = dpi.dpi_default_waves(4, B, len(ids))
    assert_plan_equals_oracle(got, dims, dtypes, 1, offs, B, len(ids), W)


@pytest.mark.parametrize("onehot", [False, True])
def test_lazy_plan_of_input_first_and_onehot_exports_in_full(onehot):
    # plans whose lookup kernel reads no partition: exported arrays still equal the oracle's
    rng = np.random.default_rng(31 + onehot)
    B, dims, dtypes = 300, [16, 16, 16], [0, 0, 0]
    lengths = np.ones((3, B), np.int64) if onehot else rng.integers(0, 50, size=(3, B))
    offs_np = G.offsets_from_lengths(lengths)
    total = int(lengths.sum())
    tabs = [torch.from_numpy((rng.standard_normal((40, 16)) * 0.01).astype(np.float32)).cuda() for _ in dims]
    ids = torch.from_numpy(rng.integers(0, 40, total).astype(np.int32)).cuda()
    offs = None if onehot else torch.from_numpy(offs_np).cuda()
    for flags in (0, dpi.DPI_FLAG_INPUT_FIRST):
        fl = FusedLookup(tabs, flags=flags)
        plan = fl.plan(offs, B, total, num_waves=97)
        out1 = fl.lookup(plan, ids, offs)
        got = dpi.dpi_plan_export(plan)
        ref = oracle.plan(dims, dtypes, 0, None if onehot else offs_np, B, total, 32, 64, 97, flags)
        for k in PLAN_KEYS:
            assert np.array_equal(got[k], ref[k]), (flags, k)
        out2 = fl.lookup(plan, ids, offs)
        assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_OK
        assert torch.equal(out1, out2)
        check([t.cpu().numpy() for t in tabs], ids.cpu().numpy(), None if onehot else offs_np, None, B, out1,
              exact=onehot)
