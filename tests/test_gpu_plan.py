"""Device plan == CPU plan oracle, bit for bit (all five workloads + edge cases)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_21101_amd import dpi
from paper_2606_21101_amd.lookup import FusedLookup
from parity import default_waves, plan_args
from synth import configs, generate as G

pytestmark = pytest.mark.gpu
KEYS = ("header", "col_base", "id_base", "bag_item_base", "bag_cost_base", "wave_item_begin")
WAVE_KEYS = ("wave_bag", "wave_bag_base", "head_first", "split_pieces", "split_last")


def check_waves(plan, ref):
    """The per-wave arrays a lookup reads, bit for bit against the oracle's closed
    forms; returns 1 when they are the planning launch's own arrays."""
    got = dpi.dpi_plan_export_waves(plan)
    for k in WAVE_KEYS:
        assert np.array_equal(got[k], ref[k]), (k, got[k][:20], ref[k][:20])
    return got["source"]


def run_plan(dims, dtypes, out_dtype, rows, lengths, onehot, C=0, K=0, W=0, flags=0):
    T, B = lengths.shape
    offs_np = G.offsets_from_lengths(lengths) if B else np.zeros((T, 1), np.int32)
    offs = None if onehot else torch.from_numpy(offs_np).cuda()
    total = int(lengths.sum())
    tabs = [torch.empty((1, d), dtype=torch.float16 if dt else torch.float32, device="cuda")
            for d, dt in zip(dims, dtypes)]
    fl = FusedLookup(tabs, None, torch.float16 if out_dtype else torch.float32, num_rows=rows,
                     chunk_rows=C, item_cost_k=K, flags=flags)
    if W == 0:
        # the library's documented default, computed here from the device's CU count
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        fill = min(16 * cus, max(-(-(T * B) // 8), min(-(-total // 32) + T * B, 8 * T)))
        W = max(fill, -(-(total + T * B) // 2048), 1)
    plan = fl.plan(offs, B, total, num_waves=W)
    got = dpi.dpi_plan_export(plan)
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_OK
    ref = oracle.plan(dims, dtypes, out_dtype, None if onehot else offs_np, B, total, C or 32, K or 64, W,
                      flags)
    for k in KEYS:
        assert np.array_equal(got[k], ref[k]), (k, got[k][:20], ref[k][:20])
    got["source"] = check_waves(plan, ref)
    return got


@pytest.mark.parametrize("key,batch", [(1, None), (2, None), (3, None), (4, None),
                                       (5, 1), (5, 16), (5, 128), (5, 512), (5, 4096)])
def test_plan_parity_configs(key, batch):
    cfg = configs.get(key, batch=batch)
    lengths = G.bag_lengths(cfg)
    dims, dtypes, out_dtype = plan_args(cfg)
    rows = G.table_sizes(cfg)
    W = default_waves(cfg, int(lengths.sum()))
    got = run_plan(dims, dtypes, out_dtype, rows, lengths, cfg.all_onehot, W=W)
    print(f"cfg{key} B={cfg.batch}: W={got['header'][3]} N={got['header'][9]} S={got['header'][10]} "
          f"split={got['header'][12]} partition from the planning launch: {got['source']}")
    # an explicit wave count: the planning launch writes the partition (one-hot
    # batches of one row class excepted: their lookup kernel reads none)
    assert got["source"] == (0 if (cfg.all_onehot and len(set(dims)) == 1) else 1)
    for W2, flags in ((7, 0), (1000, dpi.DPI_FLAG_EXACT_SPLIT)):
        run_plan(dims, dtypes, out_dtype, rows, lengths, cfg.all_onehot, W=W2, flags=flags)


@pytest.mark.parametrize("case", ["all_empty", "one_long_bag", "single_table", "w1", "w_over_n", "c1",
                                  "mixed_dims", "zero_batch", "max_tables", "max_dim", "huge_wave_request",
                                  "default_waves"])
def test_plan_parity_edges(case):
    rng = np.random.default_rng(3)
    dims, dtypes, rows, lengths, kw = [16, 8], [0, 1], [100, 100], None, {}
    if case == "all_empty":
        lengths = np.zeros((2, 50), np.int64)
    elif case == "one_long_bag":
        lengths = np.array([[256], [0]], np.int64)
        kw = dict(W=64, flags=dpi.DPI_FLAG_EXACT_SPLIT)
    elif case == "single_table":
        dims, dtypes, rows = [64], [1], [1000]
        lengths = rng.integers(0, 90, size=(1, 333))
    elif case == "w1":
        lengths = rng.integers(0, 40, size=(2, 100))
        kw = dict(W=1)
    elif case == "w_over_n":
        lengths = rng.integers(0, 3, size=(2, 10))
        kw = dict(W=5000)
    elif case == "c1":
        lengths = rng.integers(0, 9, size=(2, 77))
        kw = dict(C=1, K=1, W=37, flags=dpi.DPI_FLAG_EXACT_SPLIT)
    elif case == "mixed_dims":
        dims, dtypes, rows = [3, 12, 300, 256, 4], [0, 0, 0, 0, 1], [10, 10, 10, 10, 10]
        lengths = rng.integers(0, 70, size=(5, 41))
        kw = dict(W=19)
    elif case == "zero_batch":
        lengths = np.zeros((2, 0), np.int64)
        kw = dict(W=8)
    elif case == "max_tables":                      # DPI_MAX_TABLES fields of mixed row classes
        T = dpi.DPI_MAX_TABLES
        dims = [(4, 8, 16, 32, 3)[t % 5] for t in range(T)]
        dtypes = [t % 2 for t in range(T)]
        dims = [d if (d * (2 if dt else 4)) % 4 == 0 else d + 1 for d, dt in zip(dims, dtypes)]
        rows = [50] * T
        lengths = rng.integers(0, 12, size=(T, 20))
        kw = dict(W=333)
    elif case == "max_dim":                         # DPI_MAX_DIM elements per row
        dims, dtypes, rows = [65536], [0], [4]
        lengths = np.array([[2, 0, 5]], np.int64)
        kw = dict(W=3, flags=dpi.DPI_FLAG_EXACT_SPLIT)
    elif case == "huge_wave_request":
        lengths = rng.integers(0, 40, size=(2, 100))
        kw = dict(W=1_000_000)
    elif case == "default_waves":
        lengths = rng.integers(0, 40, size=(2, 1000))
    run_plan(dims, dtypes, 0, rows, lengths.astype(np.int64), False, **kw)


def test_plan_parity_large_onehot_batch():
    """A million one-hot samples over two fields (no offsets): the plan's closed
    form for one-id bags, 2^21 bags."""
    B = 1 << 20
    lengths = np.ones((2, B), np.int64)
    got = run_plan([16, 8], [0, 0], 0, [1000, 1000], lengths, True, W=5000)
    assert got["header"][9] == 2 * B


@pytest.mark.parametrize("T,B", [(1, 1024 * 16384), (1, 1024 * 16384 + 1), (3, 6_000_000)])
def test_plan_parity_tile_counts(T, B):
    """Batches with explicit unit offsets around the largest tile count that
    plans in one launch (1024 tiles of 16,384 bags): at it, one past it, and
    beyond it, where a separate launch scans the tile sums.  The same batches
    without offsets take the closed-form one-hot plan."""
    lengths = np.ones((T, B), np.int64)
    for onehot in (False, True):
        got = run_plan([16, 8, 4][:T], [0, 1, 0][:T], 0, [1000] * T, lengths, onehot, W=4099)
        assert got["header"][9] == T * B


def test_plan_parity_many_tiles_multihot():
    """Explicit offsets over 18 M bags (about 1100 tiles): lengths 0..5, some
    empty bags, the tile-sum launch and split bags under a tight wave count."""
    rng = np.random.default_rng(11)
    lengths = rng.integers(0, 6, size=(3, 6_000_000))
    run_plan([16, 8, 64], [0, 1, 1], 1, [1000] * 3, lengths, False, W=70_001, C=2,
             flags=dpi.DPI_FLAG_EXACT_SPLIT)
    run_plan([16, 8, 64], [0, 1, 1], 1, [1000] * 3, lengths, False)


@pytest.mark.parametrize("T,B", [(1, 1_600_000), (2, 4_500_000)])
def test_plan_parity_tiles_beyond_residency(T, B):
    """One-launch plans of many tiles: about 390 tiles of 4,096 bags (every
    block resident at once), and about 550 tiles of 16,384 bags, more than the
    512 blocks of the 64-slab kernel that fit on the device together, so the
    first blocks sum the tiles of the blocks that start later.  Bags of 0..5
    ids, split bags under a tight wave count, then the default one."""
    rng = np.random.default_rng(12)
    lengths = rng.integers(0, 6, size=(T, B))
    run_plan([16, 64][:T], [0, 1][:T], 1, [1000] * T, lengths, False, W=50_001, C=2)
    run_plan([16, 64][:T], [0, 1][:T], 1, [1000] * T, lengths, False)


@pytest.mark.parametrize("B", [600, 5000])
def test_plan_parity_wide_tiles(B):
    """Tiles whose cost reaches 2^32 bytes (64 rows of 256 KiB per bag) take
    the planner's 64-bit scan; the batch mixes them with tiles that fit 32
    bits (bags of one row, and a second field of small rows).  600 bags: one
    tile; 5,000 bags: 20 tiles of 256 bags in one launch."""
    rng = np.random.default_rng(13)
    lengths = np.ones((2, B), np.int64)
    lengths[0, : B * 3 // 5] = 64
    lengths[1] = rng.integers(0, 6, size=B)
    for W, flags in ((0, 0), (977, 0), (977, dpi.DPI_FLAG_EXACT_SPLIT), (1, 0)):
        run_plan([65536, 16], [0, 1], 0, [1000, 1000], lengths, False, W=W, flags=flags)


@pytest.mark.parametrize("W", [0, 977])
def test_plan_parity_long_form_tile_sums(W):
    """Tiles whose cost lies between 2^31 and 2^32 bytes (40 rows of 256 KiB
    per bag, 256 bags per tile): their scan stays 32-bit, but their sums do
    not fit the short published form and take the long one, beside tiles in
    the short form (a second field of small rows), in one launch of 40 tiles."""
    rng = np.random.default_rng(17)
    B = 5000
    lengths = np.empty((2, B), np.int64)
    lengths[0] = 40
    lengths[1] = rng.integers(0, 6, size=B)
    run_plan([65536, 16], [0, 1], 0, [1000, 1000], lengths, False, W=W)


@pytest.mark.parametrize("flags", [0, dpi.DPI_FLAG_EXACT_SPLIT])
def test_plan_parity_boundary_products_beyond_64_bits(flags):
    """A batch whose total cost times the wave count exceeds 2^62 (one-row
    items of cost 2^31 - 1 bytes: S near 2^51, 4,096 waves), so the wave
    boundaries take the planner's 128-bit quotients instead of the 64-bit
    ones; then the same bags under 977 waves (64-bit)."""
    lengths = np.full((1, 4096), 256, np.int64)
    lengths[0, ::7] = 3
    for W in (4096, 977):
        run_plan([16], [0], 0, [1000], lengths, False, C=1, K=2**31 - 1, W=W, flags=flags)


@pytest.mark.parametrize("W", [1, 7, 26 * 4096, 1_000_000, 0])
def test_plan_onehot_closed_form_wave_counts(W):
    """The closed-form one-hot plan against the oracle at wave counts from one
    to beyond the number of bags (0: the default rule), mixed row classes."""
    rng = np.random.default_rng(5)
    dims = [int(d) for d in rng.choice([4, 8, 16, 32, 60, 128], size=26)]
    dtypes = [int(x) for x in rng.integers(0, 2, size=26)]
    dims = [d if (d * (2 if dt else 4)) % 4 == 0 else d + 1 for d, dt in zip(dims, dtypes)]
    lengths = np.ones((26, 4096), np.int64)
    run_plan(dims, dtypes, 1, [100] * 26, lengths, True, W=W)
    run_plan(dims, dtypes, 0, [100] * 26, lengths, True, W=W, K=1000)


def test_plan_onehot_null_offsets_equals_explicit():
    cfg = configs.get(2)
    lengths = G.bag_lengths(cfg)
    dims, dtypes, out_dtype = plan_args(cfg)
    rows = G.table_sizes(cfg)
    a = run_plan(dims, dtypes, out_dtype, rows, lengths, True, W=3000)
    b = run_plan(dims, dtypes, out_dtype, rows, lengths, False, W=3000)
    for k in KEYS:
        assert np.array_equal(a[k], b[k])


def test_bad_offsets_detected():
    tabs = [torch.zeros((10, 16), device="cuda")]
    fl = FusedLookup(tabs)
    for bad, total in (([1, 1, 3], 3), ([0, 3, 1], 3), ([0, 1, 3], 4)):
        offs = torch.tensor([bad], dtype=torch.int32, device="cuda")
        plan = fl.plan(offs, 2, total, num_waves=4)
        assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_ERR_BAD_OFFSETS
        out = torch.full((2, 16), 7.0, device="cuda")
        ids = torch.zeros(total, dtype=torch.int32, device="cuda")
        fl.lookup(plan, ids, offs, out)
        torch.cuda.synchronize()
        assert torch.all(out == 7.0)      # the malformed field is not written
        fl_if = FusedLookup(tabs, flags=dpi.DPI_FLAG_INPUT_FIRST)
        plan_if = fl_if.plan(offs, 2, total, num_waves=4)
        assert dpi.dpi_plan_sync_status(plan_if) == dpi.DPI_ERR_BAD_OFFSETS
        fl_if.lookup(plan_if, ids, offs, out)
        torch.cuda.synchronize()
        assert torch.all(out == 7.0)


@pytest.mark.parametrize("key", [3, 4])
def test_lookup_reads_the_exported_partition(key):
    """The default plan of the multi-hot and large workloads, as the planning
    launch wrote it and a lookup then read it: wave starts and every per-wave
    array bit for bit against the oracle, before the export plans again."""
    cfg = configs.get(key)
    lengths = G.bag_lengths(cfg)
    dims, dtypes, out_dtype = plan_args(cfg)
    offs_np = G.offsets_from_lengths(lengths)
    total = int(lengths.sum())
    tabs = [torch.empty((1, d), dtype=torch.float16, device="cuda") for d in dims]
    fl = FusedLookup(tabs, None, torch.float16, num_rows=G.table_sizes(cfg))
    plan = fl.plan(torch.from_numpy(offs_np).cuda(), cfg.batch, total)   # default wave count
    waves = dpi.dpi_plan_export_waves(plan)
    assert waves["source"] == 1
    got = dpi.dpi_plan_export(plan)
    W = int(got["header"][3])
    assert W == default_waves(cfg, total)
    ref = oracle.plan(dims, dtypes, out_dtype, offs_np, cfg.batch, total, 32, 64, W, 0)
    for k in KEYS:
        assert np.array_equal(got[k], ref[k]), k
    for k in WAVE_KEYS:
        assert np.array_equal(waves[k], ref[k]), k
    print(f"cfg{key}: W={W}, split bags {int(got['header'][12])}, "
          f"{int(np.count_nonzero(waves['head_first'] >= 0))} boundaries inside bags")


@pytest.mark.parametrize("W", [997, 20_000])
def test_exact_split_partition_as_written(W):
    """EXACT_SPLIT plans of the multi-hot workload (many bags cut between waves):
    the planning launch's own per-wave arrays against the oracle."""
    cfg = configs.get(3)
    lengths = G.bag_lengths(cfg)
    dims, dtypes, out_dtype = plan_args(cfg)
    got = run_plan(dims, dtypes, out_dtype, G.table_sizes(cfg), lengths, False, C=8, W=W,
                   flags=dpi.DPI_FLAG_EXACT_SPLIT)
    assert got["source"] == 1
    assert got["header"][12] > W // 2


def test_superseded_plan_is_refused():
    """Planning into a workspace again supersedes the plan before: the binding
    refuses a lookup or export with it, and so does the C ABI's export (the
    workspace records which plan planned into it last)."""
    import ctypes
    tabs = [torch.zeros((10, 16), device="cuda")]
    fl = FusedLookup(tabs)
    offs = torch.tensor([[0, 1, 3]], dtype=torch.int32, device="cuda")
    ids = torch.zeros(3, dtype=torch.int32, device="cuda")
    first = fl.plan(offs, 2, 3, num_waves=4)
    second = fl.plan(offs, 2, 3, num_waves=4)
    with pytest.raises(dpi.DpiError):
        fl.lookup(first, ids, offs)
    with pytest.raises(dpi.DpiError):
        dpi.dpi_plan_export(first)
    hdr = np.zeros(16, np.int64)
    st = dpi.load().dpi_plan_export(ctypes.c_void_p(first.handle),
                                    hdr.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), None, None, None, None, None)
    assert st == dpi.DPI_ERR_INVALID_ARG and "later plan" in dpi.dpi_last_error()
    fl.lookup(second, ids, offs)
    assert dpi.dpi_plan_export(second)["header"][2] == 2


@pytest.mark.parametrize("T,B,late", [(2, 100_000, False), (1, 18_000_000, False), (1, 9_000_000, False),
                                      (1, 9_000_000, True)])
def test_bad_offsets_detected_in_multi_tile_batches(T, B, late):
    """Malformed offsets seen by several threads of one tile, in batches planned
    by one launch (at most 1024 tiles; 9 M bags are more tiles than fit on the
    device at once) and by three (more): the plan must reject them.  (A
    tile's flag once summed the count of threads that saw a malformed bag into
    its malformed bit, so two such threads cleared it.)  late: the malformed
    bags sit in a tile past the first blocks' own, summed by a block that
    sums several tiles."""
    lengths = np.ones((T, B), np.int64)
    offs_np = G.offsets_from_lengths(lengths).astype(np.int32)
    at = B - 1000 if late else 1000
    offs_np[0, at + 1] = offs_np[0, at] - 1     # decreasing: bags at - 1 and at both malformed
    offs_np[0, at + 500] = offs_np[0, at + 499] - 5
    total = int(offs_np[:, -1].astype(np.int64).sum())
    tabs = [torch.zeros((10, 16), device="cuda") for _ in range(T)]
    fl = FusedLookup(tabs)
    plan = fl.plan(torch.from_numpy(offs_np).cuda(), B, total, num_waves=4096)
    assert dpi.dpi_plan_sync_status(plan) == dpi.DPI_ERR_BAD_OFFSETS


# Planner fuzz: each case draws a field count, a batch size (so that the tile
# count lands on one of the planner's paths: one tile, every tile resident,
# more tiles than resident blocks, beyond 1,024 tiles), a row width and dtype
# per field, a bag-length law (zeros, Poisson, a few long bags, rows wide
# enough to make some tiles cost 2^32 bytes), a wave count, chunk size, item
# cost and the exact-split flag; the plan is compared with the oracle's bit
# for bit, per-wave arrays included.
PLAN_FUZZ_BAGS = [1_500, 40_000, 400_000, 1_700_000, 9_000_000, 18_000_000]


@pytest.mark.parametrize("seed", range(12))
def test_plan_fuzz(seed):
    rng = np.random.default_rng(7100 + seed)
    T = int(rng.integers(1, 9))
    bags = PLAN_FUZZ_BAGS[seed % len(PLAN_FUZZ_BAGS)]
    B = max(1, bags // T)
    dims = [int(rng.choice([4, 16, 64, 128, 1024, 65536 if seed % 4 == 3 else 256])) for _ in range(T)]
    dtypes = [int(rng.integers(0, 2)) for _ in range(T)]
    law = seed % 3
    if law == 0:
        lengths = rng.integers(0, 4, size=(T, B))
    elif law == 1:
        lengths = rng.poisson(float(rng.uniform(1, 30)), size=(T, B)).clip(0, 300)
    else:
        lengths = rng.integers(0, 12, size=(T, B))
        hot = rng.integers(0, T * B, size=8)
        lengths.reshape(-1)[hot] = rng.integers(500, 5000, size=8)
    lengths = lengths.astype(np.int64)
    C = int(rng.choice([0, 1, 8, 32]))
    K = int(rng.choice([0, 1, 64, 4096]))
    W = int(rng.choice([0, 1, 977, 65_536, 400_000]))
    flags = dpi.DPI_FLAG_EXACT_SPLIT if rng.integers(0, 2) else 0
    print(f"  plan fuzz seed {seed}: T={T} B={B} dims={dims} C={C} K={K} W={W} flags={flags}", flush=True)
    run_plan(dims, dtypes, int(rng.integers(0, 2)), [1000] * T, lengths, False, C=C, K=K, W=W, flags=flags)
