"""One-launch lookups of small batches (no planning launch), against the oracle.

One-hot batches of one row class, and bag-by-bag batches of at most 64 fields
and (with offsets) at most 1024 bags per field, take one kernel per lookup:
the lookup derives each field's first id from the offsets, checks the
offsets, and pools bags of more than 4 * C ids in pieces spread over the
field's waves.  Each case is also run with an explicit wave count (the plan's
partition, planned by its own launch) against the same oracle.
"""
import numpy as np
import pytest
import torch

from paper_2606_21101_amd import dpi
from paper_2606_21101_amd.lookup import FusedLookup
from test_gpu_edges import check, random_problem, run_case

pytestmark = pytest.mark.gpu


def with_lengths(rng, tables, lens):
    """Offsets and ids (uniform over each table's rows) for a [T, B] length matrix."""
    T, B = lens.shape
    offs = np.zeros((T, B + 1), np.int32)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    ids = np.concatenate([rng.integers(0, tables[t].shape[0], int(offs[t, -1])) for t in range(T)])
    return offs, ids.astype(np.int32)


LONG_CASES = {
    # name: (B, dims, dtypes, {(field, bag): length})
    "one_bag_b1": (1, [16, 64, 8], [0, 1, 0], {(1, 0): 5000}),
    "b3_two_fields": (3, [16, 64, 8], [0, 1, 0], {(0, 1): 129, (2, 2): 700}),
    "adjacent_long_bags": (64, [32, 16], [1, 0], {(0, 10): 300, (0, 11): 131, (0, 12): 129, (0, 13): 1000}),
    "many_long_b200": (200, [16, 32, 8, 64], [0, 0, 1, 1],
                       {(t, b): 129 + 37 * ((t * 7 + b) % 11) for t in range(4) for b in range(0, 200, 9)}),
    "longest_b1024": (1024, [8, 128], [0, 1], {(0, 1023): 20000, (1, 0): 4000, (1, 512): 128, (1, 513): 129}),
}


@pytest.mark.parametrize("name", sorted(LONG_CASES))
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.float16])
def test_long_bags_pooled_in_pieces(name, out_dtype):
    B, dims, dtypes, longs = LONG_CASES[name]
    rng = np.random.default_rng(len(name) * 1000 + B)
    tables, _, offs0, _ = random_problem(rng, dims, dtypes, B, 12, rows=400)
    lens = np.diff(offs0, axis=1).astype(np.int64)
    for (t, b), n in longs.items():
        lens[t, b] = n
    offs, ids = with_lengths(rng, tables, lens)
    for pool in ([0] * len(dims), [1] * len(dims)):
        print(f"  {name} B={B} pool={pool[0]} out={out_dtype}", flush=True)
        out, st, _, _ = run_case(tables, ids, offs, pool, B, out_dtype)
        assert st == dpi.DPI_OK
        check(tables, ids, offs, pool, B, out)
        out_p, st_p, _, _ = run_case(tables, ids, offs, pool, B, out_dtype, num_waves=37)
        assert st_p == dpi.DPI_OK
        check(tables, ids, offs, pool, B, out_p)


def test_long_bags_repeated_lookups_bit_identical():
    """The last piece of a bag clears its ticket: the same plan looked up again
    (and again after another plan used the workspace) gives the same bits."""
    B, dims, dtypes, longs = LONG_CASES["adjacent_long_bags"]
    rng = np.random.default_rng(5)
    tables, _, offs0, pool = random_problem(rng, dims, dtypes, B, 12, rows=400)
    lens = np.diff(offs0, axis=1).astype(np.int64)
    for (t, b), n in longs.items():
        lens[t, b] = n
    offs, ids = with_lengths(rng, tables, lens)
    tt = [torch.from_numpy(t).cuda() for t in tables]
    fl = FusedLookup(tt, pool)
    ids_d, offs_d = torch.from_numpy(ids).cuda(), torch.from_numpy(offs).cuda()
    plan = fl.plan(offs_d, B, len(ids))
    outs = [fl.lookup(plan, ids_d, offs_d) for _ in range(3)]
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_OK
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    check(tables, ids, offs, pool, B, outs[0])
    # another plan (other lengths) in the same workspace, then this batch again
    lens2 = lens.copy()
    lens2[1, 3] = 900
    offs2, ids2 = with_lengths(rng, tables, lens2)
    plan2 = fl.plan(torch.from_numpy(offs2).cuda(), B, len(ids2))
    out2 = fl.lookup(plan2, torch.from_numpy(ids2).cuda(), torch.from_numpy(offs2).cuda())
    check(tables, ids2, offs2, pool, B, out2)
    plan3 = fl.plan(offs_d, B, len(ids))
    assert torch.equal(fl.lookup(plan3, ids_d, offs_d), outs[0])


def test_workspace_garbage_is_not_state():
    """A workspace full of arbitrary bytes: status words and tickets tagged with
    another plan's id count as clear, so nothing needs resetting first."""
    B, dims, dtypes, longs = LONG_CASES["b3_two_fields"]
    rng = np.random.default_rng(6)
    tables, _, offs0, pool = random_problem(rng, dims, dtypes, B, 12, rows=400)
    lens = np.diff(offs0, axis=1).astype(np.int64)
    for (t, b), n in longs.items():
        lens[t, b] = n
    offs, ids = with_lengths(rng, tables, lens)
    tt = [torch.from_numpy(t).cuda() for t in tables]
    fl = FusedLookup(tt, pool)
    ids_d, offs_d = torch.from_numpy(ids).cuda(), torch.from_numpy(offs).cuda()
    o = fl.opts()
    ws = fl.workspace(B, len(ids), o)
    for fill in (0xFF, 0x00, 0x5A):
        ws.fill_(fill)
        plan = dpi.dpi_plan(fl.meta, offs_d, B, len(ids), o, ws)
        out = torch.empty((B, fl.total_dim), device="cuda")
        dpi.dpi_lookup(plan, fl._table_ptrs, ids_d, offs_d, fl._pool, out)
        assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_OK
        check(tables, ids, offs, pool, B, out)


def test_status_of_one_plan_does_not_leak_into_the_next():
    rng = np.random.default_rng(7)
    tables, ids, offs, pool = random_problem(rng, [16, 8], [0, 1], 12, 6, p_empty=0.0)
    tt = [torch.from_numpy(t).cuda() for t in tables]
    fl = FusedLookup(tt, pool)
    offs_d = torch.from_numpy(offs).cuda()
    bad = ids.copy()
    bad[3] = 10_000
    plan = fl.plan(offs_d, 12, len(ids))
    fl.lookup(plan, torch.from_numpy(bad).cuda(), offs_d)
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_ERR_BAD_ID
    plan2 = fl.plan(offs_d, 12, len(ids))
    out = fl.lookup(plan2, torch.from_numpy(ids).cuda(), offs_d)
    assert dpi.dpi_plan_sync_status(plan2) == dpi.DPI_OK
    check(tables, ids, offs, pool, 12, out)
    # one-hot batch of one row class: the other one-launch kernel
    oh = np.concatenate([rng.integers(0, 50, 12) for _ in range(2)]).astype(np.int32)
    fl1 = FusedLookup([torch.from_numpy(tables[0]).cuda()] * 2, None)
    p1 = fl1.plan(None, 12, 24)
    oh_bad = oh.copy()
    oh_bad[20] = -1
    fl1.lookup(p1, torch.from_numpy(oh_bad).cuda(), None)
    assert dpi.dpi_plan_sync_status(p1) == dpi.DPI_ERR_BAD_ID
    p2 = fl1.plan(None, 12, 24)
    out1 = fl1.lookup(p2, torch.from_numpy(oh).cuda(), None)
    assert dpi.dpi_plan_sync_status(p2) == dpi.DPI_OK
    check([tables[0], tables[0]], oh, None, [0, 0], 12, out1, exact=True)


def malformed(kind, B):
    """Two fields of B bags; field 0's offsets broken as `kind` (field 1 fine)."""
    lens = np.full((2, B), 2, np.int64)
    offs = np.zeros((2, B + 1), np.int32)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    total = int(offs[:, -1].sum())
    k = B // 2
    if kind == "first_not_zero":
        offs[0] += 1
        total += 1
    elif kind == "decreasing":
        offs[0, k + 1] = offs[0, k] - 1
    elif kind == "total_mismatch":
        total += 3
    elif kind == "negative_count":
        offs[0, 1:] = -np.arange(1, B + 1)
        total = int(offs[:, -1].sum())
    return offs, total


@pytest.mark.parametrize("B", [2, 300, 1024])
@pytest.mark.parametrize("kind", ["first_not_zero", "decreasing", "total_mismatch", "negative_count"])
@pytest.mark.parametrize("query_first", [False, True])
def test_malformed_offsets_latched(B, kind, query_first):
    """Malformed offsets are reported whether the status is queried before any
    lookup (the query checks them) or after one (the lookup checks them); the
    lookup writes nothing of a field with malformed offsets."""
    offs, total = malformed(kind, B)
    tabs = [torch.zeros((10, 16), device="cuda"), torch.zeros((10, 8), device="cuda", dtype=torch.float16)]
    fl = FusedLookup(tabs)
    offs_d = torch.from_numpy(offs).cuda()
    print(f"  malformed {kind} B={B} query_first={query_first}", flush=True)
    plan = fl.plan(offs_d, B, total)
    if query_first:
        assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_ERR_BAD_OFFSETS
    out = torch.full((B, 24), 7.0, device="cuda")
    fl.lookup(plan, torch.zeros(max(total, 1), dtype=torch.int32, device="cuda"), offs_d, out)
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_ERR_BAD_OFFSETS
    assert torch.all(out[:, :16] == 7.0)


@pytest.mark.parametrize("B", [1024, 1025])
def test_batch_size_limit_both_sides(B):
    """1024 bags per field: one launch; 1025: planned by its own launch."""
    rng = np.random.default_rng(B)
    tables, ids, offs, pool = random_problem(rng, [16, 32], [0, 1], B, 20, rows=300)
    lens = np.diff(offs, axis=1).astype(np.int64)
    lens[0, 5] = 400
    offs, ids = with_lengths(rng, tables, lens)
    out, st, _, _ = run_case(tables, ids, offs, pool, B)
    assert st == dpi.DPI_OK
    check(tables, ids, offs, pool, B, out)


@pytest.mark.parametrize("T", [64, 65])
def test_field_count_limit_both_sides(T):
    """64 fields: one launch; 65: the planning launch writes the fields' info."""
    rng = np.random.default_rng(T)
    dims = [8 * (1 + t % 4) for t in range(T)]
    dtypes = [t % 2 for t in range(T)]
    tables, ids, offs, pool = random_problem(rng, dims, dtypes, 9, 5, rows=30)
    out, st, _, _ = run_case(tables, ids, offs, pool, 9)
    assert st == dpi.DPI_OK
    check(tables, ids, offs, pool, 9, out)
    oh = np.concatenate([rng.integers(0, 30, 9) for _ in range(T)]).astype(np.int32)
    out1, st1, _, _ = run_case(tables, oh, None, pool, 9)
    assert st1 == dpi.DPI_OK
    check(tables, oh, None, pool, 9, out1, exact=True)


@pytest.mark.parametrize("B", [1, 1000])
def test_empty_batches_and_empty_fields(B):
    """Every bag empty (no ids at all), then one field without ids among
    others: zeros where there is nothing to pool, status clean."""
    rng = np.random.default_rng(B + 3)
    tables, _, _, pool = random_problem(rng, [16, 64, 8], [0, 1, 0], B, 4, rows=50)
    lens = np.zeros((3, B), np.int64)
    offs, ids = with_lengths(rng, tables, lens)
    out, st, _, _ = run_case(tables, ids, offs, pool, B)
    assert st == dpi.DPI_OK
    assert torch.all(out == 0)
    lens = rng.integers(0, 6, size=(3, B))
    lens[1] = 0
    offs, ids = with_lengths(rng, tables, lens)
    out, st, _, _ = run_case(tables, ids, offs, pool, B)
    assert st == dpi.DPI_OK
    check(tables, ids, offs, pool, B, out)


def test_sixty_four_fields_one_sample():
    """The widest one-launch batch at B = 1: 64 fields of every row class."""
    rng = np.random.default_rng(64)
    dims = [4 * (1 << (t % 7)) for t in range(64)]          # 16 .. 1024-byte fp32 rows
    dtypes = [0] * 64
    tables, ids, offs, pool = random_problem(rng, dims, dtypes, 1, 30, rows=20)
    out, st, _, _ = run_case(tables, ids, offs, pool, 1)
    assert st == dpi.DPI_OK
    check(tables, ids, offs, pool, 1, out)
