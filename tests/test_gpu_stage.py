"""One-hot input consolidation on the GPU (dpi_stage_onehot) against the
oracle, bit for bit, and end to end through the lookup."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_21101_amd import dpi
from paper_2606_21101_amd.lookup import FusedLookup

pytestmark = pytest.mark.gpu

XT = {dpi.DPI_X_F32: (np.float32, torch.float32), dpi.DPI_X_I64: (np.int64, torch.int64),
      dpi.DPI_X_I32: (np.int32, torch.int32)}


def stage(x_np, x_dtype, T):
    B, stride = x_np.shape
    host = torch.empty((B, stride), dtype=XT[x_dtype][1], pin_memory=True)
    host.copy_(torch.from_numpy(x_np))
    staging = torch.empty(max(1, B * stride * host.element_size()), dtype=torch.uint8, device="cuda")
    ids = torch.full((max(1, T * B),), 12345, dtype=torch.int32, device="cuda")
    dpi.dpi_stage_onehot(host, x_dtype, B, T, stride, staging, ids)
    torch.cuda.synchronize()
    return ids[: T * B].cpu().numpy()


def features(rng, B, stride, x_dtype, rows=1000):
    x = rng.integers(0, rows, size=(B, stride)).astype(np.float64)
    bad = rng.random((B, stride)) < 0.05
    if x_dtype == dpi.DPI_X_F32:
        junk = rng.choice([-1.0, 0.5, 2.0 ** 31, np.nan, np.inf, -0.0, 1e10], size=int(bad.sum()))
    else:
        junk = rng.choice([-1, -2 ** 40, 2 ** 31, 2 ** 31 - 1, 2 ** 33], size=int(bad.sum())).astype(np.float64)
    x[bad] = junk
    if x_dtype == dpi.DPI_X_I32:
        x = np.clip(x, -2 ** 31, 2 ** 31 - 1)
    return x.astype(XT[x_dtype][0])


@pytest.mark.parametrize("x_dtype", [dpi.DPI_X_F32, dpi.DPI_X_I64, dpi.DPI_X_I32])
@pytest.mark.parametrize("B,T,extra", [(1, 1, 0), (1, 39, 0), (63, 13, 2), (64, 64, 0), (65, 65, 1),
                                       (1000, 26, 13), (4096, 39, 0), (300, 130, 5)])
def test_stage_matches_oracle(x_dtype, B, T, extra):
    rng = np.random.default_rng(B * 1000 + T * 10 + x_dtype)
    x = features(rng, B, T + extra, x_dtype)
    got = stage(x, x_dtype, T)
    assert np.array_equal(got, oracle.stage_onehot(x, T))


def test_stage_then_lookup_equals_direct_ids():
    rng = np.random.default_rng(9)
    B, T, D, rows = 777, 13, 16, 500
    tables = [torch.from_numpy((rng.standard_normal((rows, D)) * 0.01).astype(np.float32)).cuda() for _ in range(T)]
    x = rng.integers(0, rows, size=(B, T + 2)).astype(np.float32)
    ids_staged = torch.from_numpy(stage(x, dpi.DPI_X_F32, T)).cuda()
    ids_direct = torch.from_numpy(np.ascontiguousarray(x[:, :T].T.astype(np.int32)).reshape(-1)).cuda()
    fl = FusedLookup(tables)
    assert torch.equal(fl(ids_staged, None, B), fl(ids_direct, None, B))


def test_stage_rejects_bad_arguments():
    staging = torch.empty(64, dtype=torch.uint8, device="cuda")
    ids = torch.empty(8, dtype=torch.int32, device="cuda")
    x = torch.zeros((2, 4), dtype=torch.float32, pin_memory=True)
    for args, code in (((x, 7, 2, 4, 4), dpi.DPI_ERR_INVALID_ARG),
                       ((x, dpi.DPI_X_F32, 2, 5, 4), dpi.DPI_ERR_INVALID_ARG),
                       ((x, dpi.DPI_X_I64, 2, 4, 8), dpi.DPI_ERR_INVALID_ARG)):   # staging too small
        with pytest.raises(dpi.DpiError) as ei:
            dpi.dpi_stage_onehot(*args, staging, ids)
        assert ei.value.status == code
    dpi.dpi_stage_onehot(x, dpi.DPI_X_F32, 0, 4, 4, staging, ids)    # empty batch: nothing to do


def stage_csr(packed_np, x_dtype, T, B, n_ids):
    host = torch.empty(len(packed_np), dtype=XT[x_dtype][1], pin_memory=True)
    host.copy_(torch.from_numpy(packed_np))
    staging = torch.empty(max(16, len(packed_np) * host.element_size()), dtype=torch.uint8, device="cuda")
    offs = torch.full((T, B + 1), 777, dtype=torch.int32, device="cuda")
    ids = torch.full((max(1, n_ids),), 777, dtype=torch.int32, device="cuda")
    dpi.dpi_stage_csr(host, x_dtype, T, B, n_ids, staging, offs, ids)
    torch.cuda.synchronize()
    return offs.cpu().numpy(), ids[:n_ids].cpu().numpy()


@pytest.mark.parametrize("x_dtype", [dpi.DPI_X_F32, dpi.DPI_X_I64, dpi.DPI_X_I32])
@pytest.mark.parametrize("T,B", [(1, 1), (39, 16), (26, 512), (3, 5000)])
def test_stage_csr_matches_oracle(x_dtype, T, B):
    rng = np.random.default_rng(T * 7 + B)
    lens = rng.integers(0, 30, size=(T, B))
    offs = np.zeros((T, B + 1), np.int64)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    n_ids = int(offs[:, -1].sum())
    ids = rng.integers(0, 1 << 20, size=n_ids)
    packed = np.concatenate([offs.reshape(-1), ids]).astype(np.float64)
    bad = rng.random(len(packed)) < 0.02
    packed[bad] = -5 if x_dtype != dpi.DPI_X_F32 else 2.5
    packed = packed.astype(XT[x_dtype][0])
    got_o, got_i = stage_csr(packed, x_dtype, T, B, n_ids)
    want_o, want_i = oracle.stage_csr(packed, T, B, n_ids)
    assert np.array_equal(got_o, want_o) and np.array_equal(got_i, want_i)


def test_stage_csr_then_lookup_equals_direct():
    rng = np.random.default_rng(21)
    T, B, D, rows = 5, 300, 32, 400
    tables = [torch.from_numpy((rng.standard_normal((rows, D)) * 0.01).astype(np.float16)).cuda() for _ in range(T)]
    lens = rng.integers(0, 12, size=(T, B))
    offs = np.zeros((T, B + 1), np.int64)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    n_ids = int(offs[:, -1].sum())
    ids = rng.integers(0, rows, size=n_ids)
    got_o, got_i = stage_csr(np.concatenate([offs.reshape(-1), ids]), dpi.DPI_X_I64, T, B, n_ids)
    fl = FusedLookup(tables, [0, 1, 0, 1, 0])
    a = fl(torch.from_numpy(got_i).cuda(), torch.from_numpy(got_o).cuda(), B)
    b = fl(torch.from_numpy(ids.astype(np.int32)).cuda(), torch.from_numpy(offs.astype(np.int32)).cuda(), B)
    assert torch.equal(a, b)


# --- the staged CSR read by the lookup itself (dpi_lookup_csr) --------------

def csr_problem(rng, B, dims, dtypes, rows=400, long_bag=0):
    T = len(dims)
    tables = [torch.from_numpy((rng.standard_normal((rows, d)) * 0.01).astype(np.float16 if dt else np.float32))
              .cuda() for d, dt in zip(dims, dtypes)]
    lens = rng.integers(0, 25, size=(T, B))
    if long_bag:
        lens[T // 2, B // 2] = long_bag
    offs = np.zeros((T, B + 1), np.int64)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    n_ids = int(offs[:, -1].sum())
    ids = rng.integers(0, rows, size=n_ids)
    return tables, offs, ids, n_ids


def lookup_csr(tables, pool, packed_np, x_dtype, B, n_ids, out_dtype=torch.float32):
    """dpi_plan over not-yet-written offsets, then dpi_lookup_csr: returns the
    output, the converted offsets and ids, and the status."""
    T = len(tables)
    host = torch.empty(len(packed_np), dtype=XT[x_dtype][1], pin_memory=True)
    host.copy_(torch.from_numpy(packed_np))
    staging = torch.empty(max(16, len(packed_np) * host.element_size()), dtype=torch.uint8, device="cuda")
    offs = torch.full((T, B + 1), 777, dtype=torch.int32, device="cuda")
    ids = torch.full((max(1, n_ids),), 777, dtype=torch.int32, device="cuda")
    fl = FusedLookup(tables, pool, out_dtype)
    plan = fl.plan(offs, B, n_ids)
    out = torch.full((B, fl.total_dim), float("nan"), dtype=out_dtype, device="cuda")
    dpi.dpi_lookup_csr(plan, host, x_dtype, staging, fl._table_ptrs, fl._pool, offs, ids, out)
    st = dpi.dpi_plan_sync_status(plan)
    return out, offs.cpu().numpy(), ids[:n_ids].cpu().numpy(), st


@pytest.mark.parametrize("x_dtype", [dpi.DPI_X_F32, dpi.DPI_X_I64, dpi.DPI_X_I32])
@pytest.mark.parametrize("B,long_bag", [(1, 0), (16, 0), (128, 0), (512, 0), (37, 700), (1024, 3000)])
def test_lookup_csr_equals_stage_then_lookup(x_dtype, B, long_bag):
    """One copy and one kernel: the converted offsets and ids bit for bit as
    the oracle converts them, and the output bit for bit as dpi_stage_csr then
    dpi_lookup gives it (the same kernel arithmetic), long bags included."""
    rng = np.random.default_rng(B * 10 + x_dtype + long_bag)
    dims, dtypes = [8, 16, 32, 64, 16, 8], [0, 0, 0, 0, 1, 1]
    tables, offs, ids, n_ids = csr_problem(rng, B, dims, dtypes, long_bag=long_bag)
    packed = np.concatenate([offs.reshape(-1), ids]).astype(XT[x_dtype][0])
    pool = [0, 1, 0, 1, 0, 1]
    print(f"  lookup_csr x_dtype={x_dtype} B={B} long={long_bag}", flush=True)
    out, got_o, got_i, st = lookup_csr(tables, pool, packed, x_dtype, B, n_ids)
    assert st == dpi.DPI_OK
    want_o, want_i = oracle.stage_csr(packed, len(dims), B, n_ids)
    assert np.array_equal(got_o, want_o) and np.array_equal(got_i, want_i)
    so, si = stage_csr(packed, x_dtype, len(dims), B, n_ids)
    ref = FusedLookup(tables, pool)(torch.from_numpy(si).cuda(), torch.from_numpy(so).cuda(), B)
    assert torch.equal(out.view(torch.int32), ref.view(torch.int32))


def test_lookup_csr_reports_bad_ids_and_offsets():
    rng = np.random.default_rng(5)
    B = 40
    tables, offs, ids, n_ids = csr_problem(rng, B, [16, 32], [0, 1])
    packed = np.concatenate([offs.reshape(-1), ids]).astype(np.float64)
    packed[2 * (B + 1) + 3] = 2.5                      # an id that is not an integer
    out, _, got_i, st = lookup_csr(tables, None, packed.astype(np.float32), dpi.DPI_X_F32, B, n_ids)
    assert st == dpi.DPI_ERR_BAD_ID and got_i[3] == -1
    bad = np.concatenate([offs.reshape(-1), ids]).astype(np.int64)
    bad[5] = -3                                        # an offset that becomes -1
    _, got_o, _, st = lookup_csr(tables, None, bad, dpi.DPI_X_I64, B, n_ids)
    assert st == dpi.DPI_ERR_BAD_OFFSETS and got_o[0, 5] == -1


def test_lookup_csr_needs_a_one_launch_plan():
    rng = np.random.default_rng(6)
    B = 2000                                           # more than 1024 bags per field: planned by its own launch
    tables, offs, ids, n_ids = csr_problem(rng, B, [16], [0])
    packed = np.concatenate([offs.reshape(-1), ids]).astype(np.int64)
    with pytest.raises(dpi.DpiError) as e:
        lookup_csr(tables, None, packed, dpi.DPI_X_I64, B, n_ids)
    assert e.value.status == dpi.DPI_ERR_UNSUPPORTED
