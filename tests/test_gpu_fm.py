"""Second-order FM term on the GPU (dpi_fm_second_order) against the oracle.

Inputs are seeded synthetic blocks made on the host (values ~ 0.01 * N(0,1),
as the tables), copied to the device; the oracle reads the same host array.
Tolerance, from the fp32 summation bound: |y - r| <= (2T + D + 8) * 2^-24 * mag
with mag = 1/2 * sum_c ((sum_t |e|)^2 + sum_t e^2).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_21101_amd import dpi

pytestmark = pytest.mark.gpu


def block(rng, B, T, D, stride, dtype):
    return (rng.standard_normal((B, stride)) * 0.01).astype(dtype)


def run_fm(e_host, T, D, offset_elems=0):
    dt = dpi.DPI_F16 if e_host.dtype == np.float16 else dpi.DPI_F32
    B, stride = e_host.shape
    flat = torch.zeros(B * stride + offset_elems, dtype=torch.from_numpy(e_host[:0]).dtype, device="cuda")
    flat[offset_elems:] = torch.from_numpy(e_host.reshape(-1)).cuda()
    out = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
    emb = flat[offset_elems:]
    dpi.dpi_fm_second_order(emb, dt, B, T, D, stride, out)
    torch.cuda.synchronize()
    return out.double().cpu().numpy()


def check(y, e_host, T, D):
    ref, mag = oracle.fm_second_order(e_host, T, D)
    tol = (2 * T + D + 8) * 2.0 ** -24
    err = np.abs(y - ref)
    bad = err > tol * mag
    assert not bad.any(), f"T={T} D={D}: max err/mag {np.max(err / np.maximum(mag, 1e-300)):.3g} > {tol:.3g}"
    return float(np.max(err / np.maximum(mag, 1e-300))) if len(y) else 0.0


@pytest.mark.parametrize("T,D,dtype", [
    (26, 64, np.float16),      # multi-hot workload's block: 128-byte rows, vector path
    (100, 128, np.float16),    # large workload's block: 256-byte rows
    (26, 60, np.float32),      # 240-byte rows: 16 lanes per row, 15 active
    (39, 16, np.float32), (2, 4, np.float32), (1, 8, np.float16),
    (7, 256, np.float32),      # 1024-byte rows: a whole wave per row
    (5, 3, np.float32), (9, 300, np.float16), (3, 1, np.float16),   # column path
])
def test_fm_shapes(T, D, dtype):
    rng = np.random.default_rng(T * 1000 + D)
    for B, extra in ((1, 0), (37, 0), (1000, 8)):
        e = block(rng, B, T, D, T * D + extra, dtype)
        check(run_fm(e, T, D), e, T, D)


def test_fm_unaligned_block_takes_column_path():
    rng = np.random.default_rng(7)
    T, D = 26, 64
    e = block(rng, 100, T, D, T * D + 3, np.float16)        # odd stride: rows not 16-byte aligned
    check(run_fm(e, T, D), e, T, D)
    e2 = block(rng, 100, T, D, T * D, np.float16)
    check(run_fm(e2, T, D, offset_elems=1), e2, T, D)        # block start not 16-byte aligned


def test_fm_large_batch_and_determinism():
    rng = np.random.default_rng(11)
    T, D, B = 100, 128, 8192
    e = block(rng, B, T, D, T * D, np.float16)
    y1 = run_fm(e, T, D)
    y2 = run_fm(e, T, D)
    assert np.array_equal(y1, y2)
    check(y1, e, T, D)


def test_fm_zero_batch_and_errors():
    out = torch.zeros(1, dtype=torch.float32, device="cuda")
    dpi.dpi_fm_second_order(None, dpi.DPI_F32, 0, 3, 4, 12, None)        # nothing to do
    emb = torch.zeros(24, dtype=torch.float32, device="cuda")
    for args, code in (((emb, dpi.DPI_F32, 2, 3, 4, 11, out), dpi.DPI_ERR_INVALID_ARG),
                       ((emb, 5, 2, 3, 4, 12, out), dpi.DPI_ERR_INVALID_ARG),
                       ((None, dpi.DPI_F32, 2, 3, 4, 12, out), dpi.DPI_ERR_INVALID_ARG)):
        with pytest.raises(dpi.DpiError) as ei:
            dpi.dpi_fm_second_order(*args)
        assert ei.value.status == code
