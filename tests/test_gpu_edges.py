"""Edge cases of the fused lookup on the GPU, each against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_21101_amd import dpi
from paper_2606_21101_amd.lookup import FusedLookup
from parity import check_outputs

pytestmark = pytest.mark.gpu


def random_problem(rng, dims, dtypes, B, max_len, rows=50, p_empty=0.1):
    T = len(dims)
    tables = []
    for d, dt in zip(dims, dtypes):
        v = rng.standard_normal((rows, d)) * 0.01
        tables.append(v.astype(np.float16 if dt else np.float32))
    lens = rng.integers(0, max_len + 1, size=(T, B))
    lens[rng.random((T, B)) < p_empty] = 0
    offs = np.zeros((T, B + 1), np.int32)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    ids = np.concatenate([rng.integers(0, rows, size=int(offs[t, -1])) for t in range(T)]).astype(np.int32)
    pool = [int(x) for x in rng.integers(0, 2, T)]
    return tables, ids, offs, pool


def run_case(tables, ids, offs, pool, B, out_dtype=torch.float32, **kw):
    tt = [torch.from_numpy(t).cuda() for t in tables]
    fl = FusedLookup(tt, pool, out_dtype, **{k: v for k, v in kw.items() if k in ("chunk_rows", "flags")})
    ids_d = torch.from_numpy(ids).cuda()
    offs_d = None if offs is None else torch.from_numpy(offs).cuda()
    plan = fl.plan(offs_d, B, len(ids), num_waves=kw.get("num_waves", 0))
    out = fl.lookup(plan, ids_d, offs_d)
    st = dpi.dpi_plan_sync_status(plan)
    return out, st, fl, plan


def check(tables, ids, offs, pool, B, out, exact=False):
    dims = [t.shape[1] for t in tables]
    ref, mag = oracle.lookup(dims, tables, ids, offs, pool, B)
    f16 = any(t.dtype == np.float16 for t in tables)
    return check_outputs(out.double().cpu().numpy(), ref, mag, f16, out.dtype == torch.float16, exact=exact)


@pytest.mark.parametrize("dims,dtypes", [
    ([3, 5, 7], [0, 0, 0]),            # 12/20/28-byte rows: general path
    ([6, 2, 10], [1, 1, 1]),           # fp16 rows of 12/4/20 bytes: general path
    ([12, 48, 24], [0, 1, 1]),         # rows of 48/96/48 bytes: lanes rounded up to a power of two
    ([300], [0]),                      # 1200-byte rows: several column passes
    ([256, 512], [0, 1]),              # 1024-byte rows: 64 lanes per row
    ([4, 8, 16, 32, 64, 128], [0, 1, 0, 1, 0, 1]),
])
def test_row_shapes(dims, dtypes):
    rng = np.random.default_rng(sum(dims))
    tables, ids, offs, pool = random_problem(rng, dims, dtypes, 37, 70)
    for flags, W in ((0, 0), (dpi.DPI_FLAG_EXACT_SPLIT, 53), (dpi.DPI_FLAG_LINEAR_BLOCKS, 0),
                     (dpi.DPI_FLAG_INPUT_FIRST, 0)):
        for od in (torch.float32, torch.float16):
            out, st, _, _ = run_case(tables, ids, offs, pool, 37, od, flags=flags, num_waves=W, chunk_rows=8)
            assert st == dpi.DPI_OK
            check(tables, ids, offs, pool, 37, out)


def test_all_bags_empty_and_zero_batch():
    rng = np.random.default_rng(1)
    tables, _, _, pool = random_problem(rng, [16, 8], [0, 1], 20, 3)
    offs = np.zeros((2, 21), np.int32)
    ids = np.zeros(0, np.int32)
    out, st, _, _ = run_case(tables, ids, offs, pool, 20)
    assert st == dpi.DPI_OK
    assert torch.all(out == 0)
    out_if, st_if, _, _ = run_case(tables, ids, offs, pool, 20, flags=dpi.DPI_FLAG_INPUT_FIRST)
    assert st_if == dpi.DPI_OK
    assert torch.all(out_if == 0)
    out0, st0, _, _ = run_case(tables, ids, np.zeros((2, 1), np.int32), pool, 0)
    assert st0 == dpi.DPI_OK and out0.shape == (0, 24)


def test_single_long_bag_split_over_many_waves():
    rng = np.random.default_rng(2)
    tables, _, _, _ = random_problem(rng, [64], [1], 1, 1, rows=500)
    ids = rng.integers(0, 500, size=256).astype(np.int32)
    offs = np.array([[0, 256]], np.int32)
    for pool in ([0], [1]):
        for W, C in ((64, 4), (8, 32), (300, 1)):
            out, st, fl, plan = run_case(tables, ids, offs, pool, 1, chunk_rows=C, num_waves=W,
                                         flags=dpi.DPI_FLAG_EXACT_SPLIT)
            hdr = dpi.dpi_plan_export(plan)["header"]
            assert hdr[12] == 1              # the one bag is split
            check(tables, ids, offs, pool, 1, out)


def test_onehot_null_offsets_bit_exact():
    rng = np.random.default_rng(4)
    tables, _, _, pool = random_problem(rng, [16, 32, 8], [0, 0, 0], 300, 1)
    ids = np.concatenate([rng.integers(0, 50, 300) for _ in range(3)]).astype(np.int32)
    out, st, _, _ = run_case(tables, ids, None, pool, 300)
    assert st == dpi.DPI_OK
    check(tables, ids, None, pool, 300, out, exact=True)


def test_out_of_range_ids_reported_and_skipped():
    rng = np.random.default_rng(5)
    tables, ids, offs, pool = random_problem(rng, [16, 8], [0, 0], 40, 6, p_empty=0.0)
    bad_ids = ids.copy()
    bad_ids[3] = -1
    bad_ids[len(ids) - 2] = 50            # == num_rows
    out, st, _, _ = run_case(tables, bad_ids, offs, pool, 40)
    assert st == dpi.DPI_ERR_BAD_ID
    out_if, st_if, _, _ = run_case(tables, bad_ids, offs, pool, 40, flags=dpi.DPI_FLAG_INPUT_FIRST)
    assert st_if == dpi.DPI_ERR_BAD_ID
    # the oracle's view: out-of-range ids contribute nothing (its status is BAD_ID)
    fixed = bad_ids.copy()
    tables_z = [np.concatenate([t, np.zeros((1, t.shape[1]), t.dtype)]) for t in tables]
    fixed[fixed < 0] = 50
    ref, mag = oracle.lookup([16, 8], tables_z, fixed, offs, [0, 0], 40)
    sums = out.double().cpu().numpy()
    # compare only sum-pooled columns (mean divides by the full length in both)
    out_s, _, _, _ = run_case(tables, bad_ids, offs, [0, 0], 40)
    check_outputs(out_s.double().cpu().numpy(), ref, mag, False, False)
    out_s2, _, _, _ = run_case(tables, bad_ids, offs, [0, 0], 40, flags=dpi.DPI_FLAG_INPUT_FIRST)
    check_outputs(out_s2.double().cpu().numpy(), ref, mag, False, False)


def test_deterministic_and_stream():
    rng = np.random.default_rng(6)
    tables, ids, offs, pool = random_problem(rng, [64, 16], [1, 0], 500, 80)
    kw = dict(flags=dpi.DPI_FLAG_EXACT_SPLIT, num_waves=97, chunk_rows=8)
    a, _, _, _ = run_case(tables, ids, offs, pool, 500, **kw)
    b, _, _, _ = run_case(tables, ids, offs, pool, 500, **kw)
    assert torch.equal(a, b)
    s = torch.cuda.Stream()
    tt = [torch.from_numpy(t).cuda() for t in tables]
    fl = FusedLookup(tt, pool, torch.float32, flags=kw["flags"], chunk_rows=8)
    ids_d, offs_d = torch.from_numpy(ids).cuda(), torch.from_numpy(offs).cuda()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        c = fl(ids_d, offs_d, 500, num_waves=97, stream=s)
    s.synchronize()
    assert torch.equal(a, c)
    check(tables, ids, offs, pool, 500, a)
    # the block-to-wave order changes where waves run, not what they compute
    kw_lin = dict(kw, flags=kw["flags"] | dpi.DPI_FLAG_LINEAR_BLOCKS)
    d, st, _, _ = run_case(tables, ids, offs, pool, 500, **kw_lin)
    assert st == dpi.DPI_OK
    assert torch.equal(a, d)


def test_max_tables_and_max_dim():
    """DPI_MAX_TABLES fields of mixed row classes (the mixed-class kernel), and
    one field of DPI_MAX_DIM elements per row (the general path, 256 KiB rows)."""
    rng = np.random.default_rng(256)
    T = dpi.DPI_MAX_TABLES
    dims = [(4, 8, 16, 32, 6)[t % 5] for t in range(T)]
    dtypes = [t % 2 for t in range(T)]
    tables, ids, offs, pool = random_problem(rng, dims, dtypes, 33, 9)
    for flags, W in ((0, 0), (dpi.DPI_FLAG_EXACT_SPLIT, 301), (dpi.DPI_FLAG_INPUT_FIRST, 0)):
        out, st, _, _ = run_case(tables, ids, offs, pool, 33, flags=flags, num_waves=W, chunk_rows=4)
        assert st == dpi.DPI_OK
        check(tables, ids, offs, pool, 33, out)
    tables, ids, offs, pool = random_problem(rng, [dpi.DPI_MAX_DIM], [0], 3, 4, rows=5)
    for flags, W in ((0, 0), (dpi.DPI_FLAG_EXACT_SPLIT, 3), (dpi.DPI_FLAG_INPUT_FIRST, 0)):
        out, st, _, _ = run_case(tables, ids, offs, pool, 3, flags=flags, num_waves=W, chunk_rows=1)
        assert st == dpi.DPI_OK
        check(tables, ids, offs, pool, 3, out)


def test_million_sample_onehot_batch():
    """2^20 one-hot samples over three fields (the one-hot kernel), sampled rows
    against the oracle, every output row written."""
    rng = np.random.default_rng(20)
    B, dims, rows = 1 << 20, [16, 32, 8], 1000
    tables = [(rng.standard_normal((rows, d)) * 0.01).astype(np.float32) for d in dims]
    ids = rng.integers(0, rows, size=3 * B).astype(np.int32)
    out, st, _, _ = run_case(tables, ids, None, [0, 1, 0], B)
    assert st == dpi.DPI_OK
    pick = np.concatenate([np.arange(100), np.arange(B // 2, B // 2 + 100), np.arange(B - 100, B)])
    sub_ids = np.concatenate([ids[t * B:(t + 1) * B][pick] for t in range(3)])
    ref, mag = oracle.lookup(dims, tables, sub_ids, None, [0, 1, 0], len(pick))
    check_outputs(out[torch.from_numpy(pick).cuda()].double().cpu().numpy(), ref, mag, False, False, exact=True)


def test_rows_beyond_2gib_of_a_table():
    """Rows whose byte offset exceeds 2^31 (buffer-descriptor range up to 4 GiB)
    and a table above 4 GiB (64-bit addressing) are read correctly."""
    rng = np.random.default_rng(9)
    for rows, dim, dtype in ((9_000_000, 128, torch.float16), (4_500_000, 256, torch.float32)):
        big = torch.empty((rows, dim), dtype=dtype, device="cuda")
        hi = torch.arange(rows - 3000, rows, device="cuda")
        lo = torch.arange(0, 3000, device="cuda")
        vals_hi = torch.from_numpy((rng.integers(-64, 64, size=(3000, dim)) / 64.0)).to(dtype).cuda()
        vals_lo = torch.from_numpy((rng.integers(-64, 64, size=(3000, dim)) / 64.0)).to(dtype).cuda()
        big[hi] = vals_hi
        big[lo] = vals_lo
        B = 500
        ids_np = np.concatenate([rng.integers(rows - 3000, rows, size=6 * B // 2), rng.integers(0, 3000, size=6 * B // 2)])
        rng.shuffle(ids_np)
        ids = torch.from_numpy(ids_np.astype(np.int32)).cuda()
        offs = torch.arange(0, 6 * B + 1, 6, dtype=torch.int32, device="cuda").view(1, -1)
        fl = FusedLookup([big], [0], torch.float32)
        out = fl(ids, offs, B)
        # reference from the two populated slices only
        table_np = np.zeros((6000, dim), dtype=np.float32)
        table_np[:3000] = vals_lo.float().cpu().numpy()
        table_np[3000:] = vals_hi.float().cpu().numpy()
        remap = np.where(ids_np >= rows - 3000, ids_np - (rows - 3000) + 3000, ids_np).astype(np.int32)
        ref, mag = oracle.lookup([dim], [table_np.astype(np.float16 if dtype == torch.float16 else np.float32)],
                                 remap, offs.cpu().numpy(), [0], B)
        check_outputs(out.double().cpu().numpy(), ref, mag, dtype == torch.float16, False)
        del big
        torch.cuda.empty_cache()


@pytest.mark.parametrize("dim,dtype", [(4, torch.float32), (128, torch.float16)])
def test_largest_buffer_table_masked_rows_read_zeros(dim, dtype):
    """A table of the largest size read through a buffer descriptor (2^32 - 16
    bytes of 16-byte rows; 2^32 - 256 bytes of 256-byte rows), pooled by the
    single-row-class kernel with bags of 3 ids, so that most row slots of a
    group are masked and loaded at the offset past the range.  The row right
    after the table (same allocation, outside the table's range) holds a
    marker that would show in every output if such a load returned data."""
    rb = dim * (4 if dtype == torch.float32 else 2)
    rows = (2 ** 32 - 16) // rb if rb == 16 else (2 ** 32) // rb - 1
    assert rows * rb <= 2 ** 32 - 16
    rng = np.random.default_rng(31)
    store = torch.empty((rows + 1, dim), dtype=dtype, device="cuda")
    store[rows] = 1000.0                                   # marker past the table
    n_set = 3000
    hi = torch.arange(rows - n_set, rows, device="cuda")
    lo = torch.arange(0, n_set, device="cuda")
    vals_hi = torch.from_numpy(rng.integers(-64, 64, size=(n_set, dim)) / 64.0).to(dtype).cuda()
    vals_lo = torch.from_numpy(rng.integers(-64, 64, size=(n_set, dim)) / 64.0).to(dtype).cuda()
    store[hi] = vals_hi
    store[lo] = vals_lo
    table = store[:rows]
    B, L = 2000, 3
    ids_np = np.concatenate([rng.integers(rows - n_set, rows, size=L * B // 2),
                             rng.integers(0, n_set, size=L * B - L * B // 2)]).astype(np.int32)
    rng.shuffle(ids_np)
    ids = torch.from_numpy(ids_np).cuda()
    offs_np = np.arange(0, L * B + 1, L, dtype=np.int32).reshape(1, -1)
    offs = torch.from_numpy(offs_np).cuda()
    fl = FusedLookup([table], [0], torch.float32)
    plan = fl.plan(offs, B, len(ids_np), num_waves=64)   # the partition: single-row-class kernel
    out = fl.lookup(plan, ids, offs)
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_OK
    small = np.zeros((2 * n_set, dim), np.float32)
    small[:n_set] = vals_lo.float().cpu().numpy()
    small[n_set:] = vals_hi.float().cpu().numpy()
    remap = np.where(ids_np >= rows - n_set, ids_np - (rows - n_set) + n_set, ids_np).astype(np.int32)
    ref, mag = oracle.lookup([dim], [small.astype(np.float16 if dtype == torch.float16 else np.float32)],
                             remap, offs_np, [0], B)
    check_outputs(out.double().cpu().numpy(), ref, mag, dtype == torch.float16, False)
    del store, table
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dim,dtype", [(64, 1), (32, 0)])
def test_row_groups_across_bag_ends(dim, dtype):
    """128-byte rows (eight lanes per row), whose row groups run on past a bag's
    end into the next bag: short bags (0..12 rows, many empty or of one row),
    sum and mean fields, explicit wave counts (the single-row-class kernel);
    the linear block order bit for bit against the default (pairs of XCDs);
    then a row holding +inf in one column, which must reach exactly the bags
    that pool that row and leave every other output bit unchanged."""
    rng = np.random.default_rng(90 + dim)
    T, B, rows = 3, 3000, 200
    dims, dtypes = [dim] * T, [dtype] * T
    tables = [(rng.standard_normal((rows, dim)) * 0.01).astype(np.float16 if dtype else np.float32)
              for _ in range(T)]
    lens = rng.integers(0, 13, size=(T, B))
    lens[rng.random((T, B)) < 0.15] = 0
    lens[rng.random((T, B)) < 0.10] = 1
    offs = np.zeros((T, B + 1), np.int32)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    ids = np.concatenate([rng.integers(0, rows, size=int(offs[t, -1])) for t in range(T)]).astype(np.int32)
    pool = [0, 1, 0]
    for W in (97, 3001):
        for od in (torch.float32, torch.float16):
            out, st, _, _ = run_case(tables, ids, offs, pool, B, od, num_waves=W)
            assert st == dpi.DPI_OK
            check(tables, ids, offs, pool, B, out)
    base, _, _, _ = run_case(tables, ids, offs, pool, B, torch.float32, num_waves=97)
    # rows of at most 128 bytes: pairs of XCDs share each range of waves; the
    # linear block order must give the same bits
    lin, st, _, _ = run_case(tables, ids, offs, pool, B, torch.float32, num_waves=97,
                             flags=dpi.DPI_FLAG_LINEAR_BLOCKS)
    assert st == dpi.DPI_OK and torch.equal(lin, base)
    hot_row, col = 5, 3
    tables_inf = [t.copy() for t in tables]
    tables_inf[1][hot_row, col] = np.inf
    out, st, _, _ = run_case(tables_inf, ids, offs, pool, B, torch.float32, num_waves=97)
    assert st == dpi.DPI_OK
    got, ref = out.cpu().numpy(), base.cpu().numpy()
    lo = int(offs[0, -1])
    seg = ids[lo: lo + int(offs[1, -1])]
    has = np.array([np.any(seg[offs[1, b]: offs[1, b + 1]] == hot_row) for b in range(B)])
    c = dim + col                     # field 1's column
    assert has.any() and np.all(np.isposinf(got[has, c]))
    keep = np.ones(got.shape, bool)
    keep[has, c] = False
    assert np.array_equal(got[keep], ref[keep])
