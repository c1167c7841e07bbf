"""Two-stream scheduling (Algorithm 2, §IV-E) and the interaction head on the
GPU: the enqueue order of each mode, and the cross network + MLP forward
against the fp64 oracle in every mode."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2606_21101_amd import dpi

pytestmark = pytest.mark.gpu


def recording_ops(n, module, log):
    ops, keep = [], []
    for i in range(n):
        def fn(ctx, stream, i=i):
            log.append((module, i, stream))
            return dpi.DPI_OK
        cb = dpi.DPI_OP_FN(fn)
        keep.append(cb)
        ops.append(dpi.dpi_op(cb, None))
    return ops, keep


@pytest.mark.parametrize("ne,ni", [(3, 5), (4, 4), (6, 1), (0, 3)])
def test_enqueue_order_and_streams(ne, ni):
    se, si = torch.cuda.Stream(), torch.cuda.Stream()
    after = torch.cuda.current_stream()
    for mode in (dpi.DPI_SCHED_BREADTH_FIRST, dpi.DPI_SCHED_DEPTH_FIRST, dpi.DPI_SCHED_ONE_STREAM):
        log = []
        eo, k1 = recording_ops(ne, "E", log)
        io, k2 = recording_ops(ni, "I", log)
        dpi.dpi_launch_two_streams(eo, io, mode, se, si, after)
        torch.cuda.synchronize()
        order = [(m, i) for m, i, _ in log]
        if mode == dpi.DPI_SCHED_BREADTH_FIRST:
            assert order == oracle.breadth_first_order(ne, ni)
        else:
            assert order == [("E", i) for i in range(ne)] + [("I", j) for j in range(ni)]
        streams = {m: {s for mm, _, s in log if mm == m} for m in ("E", "I")}
        if ne:
            assert streams["E"] == {se.cuda_stream}
        if ni:
            assert streams["I"] == ({se.cuda_stream} if mode == dpi.DPI_SCHED_ONE_STREAM else {si.cuda_stream})


def make_head(rng, B, d, n_cross, mlp_dims):
    cw = [torch.from_numpy((rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)).cuda() for _ in range(n_cross)]
    cb = [torch.from_numpy((rng.standard_normal(d) * 0.1).astype(np.float32)).cuda() for _ in range(n_cross)]
    mw, mb, prev = [], [], d
    for h in mlp_dims:
        mw.append(torch.from_numpy((rng.standard_normal((h, prev)) / np.sqrt(prev)).astype(np.float32)).cuda())
        mb.append(torch.from_numpy((rng.standard_normal(h) * 0.1).astype(np.float32)).cuda())
        prev = h
    return dpi.DcnHead(B, d, cw, cb, mw, mb), cw, cb, mw, mb


@pytest.mark.parametrize("B,d,n_cross,mlp_dims", [(300, 64, 2, [128, 32]), (1000, 416, 3, [512, 256, 130]),
                                                  (7, 13, 1, [5])])
def test_dcn_forward_all_modes(B, d, n_cross, mlp_dims):
    rng = np.random.default_rng(B + d)
    head, cw, cb, mw, mb = make_head(rng, B, d, n_cross, mlp_dims)
    x0_np = (rng.standard_normal((B, d)) * 0.5).astype(np.float32)
    x0 = torch.from_numpy(x0_np).cuda()
    ref_x, ref_h, mag_x, mag_h = oracle.dcn_forward(x0_np, [w.cpu().numpy() for w in cw], [b.cpu().numpy() for b in cb],
                                                    [w.cpu().numpy() for w in mw], [b.cpu().numpy() for b in mb])
    tol_x = n_cross * (d + 8) * 2.0 ** -24
    dims = [d] + mlp_dims
    tol_h = sum(k + 8 for k in dims[:-1]) * 2.0 ** -24
    se, si = torch.cuda.Stream(), torch.cuda.Stream()
    after = torch.cuda.current_stream()
    outs = []
    for mode in (dpi.DPI_SCHED_BREADTH_FIRST, dpi.DPI_SCHED_DEPTH_FIRST, dpi.DPI_SCHED_ONE_STREAM):
        oc = torch.full((B, d), float("nan"), device="cuda")
        om = torch.full((B, mlp_dims[-1]), float("nan"), device="cuda")
        marks = torch.zeros(2, dtype=torch.int64, device="cuda")
        head.forward(x0, oc, om, mode, se, si, after, marks)
        torch.cuda.synchronize()
        yx, yh = oc.double().cpu().numpy(), om.double().cpu().numpy()
        assert np.all(np.abs(yx - ref_x) <= tol_x * mag_x + 1e-30), f"cross, mode {mode}"
        assert np.all(np.abs(yh - ref_h) <= tol_h * mag_h + 1e-30), f"mlp, mode {mode}"
        assert torch.all(marks > 0)
        outs.append((oc, om))
    for oc, om in outs[1:]:       # the order of enqueueing changes nothing computed
        assert torch.equal(oc, outs[0][0]) and torch.equal(om, outs[0][1])


def test_dcn_forward_waits_for_after_stream():
    rng = np.random.default_rng(3)
    B, d = 2048, 64
    head, *_ = make_head(rng, B, d, 2, [64])
    x0 = torch.zeros((B, d), device="cuda")
    after = torch.cuda.Stream()
    se, si = torch.cuda.Stream(), torch.cuda.Stream()
    src = torch.from_numpy((rng.standard_normal((B, d))).astype(np.float32)).cuda()
    torch.cuda.synchronize()
    with torch.cuda.stream(after):
        for _ in range(20):                       # queue some work that writes x0 last
            x0.copy_(src)
    oc1 = torch.empty((B, d), device="cuda")
    om1 = torch.empty((B, 64), device="cuda")
    head.forward(x0, oc1, om1, dpi.DPI_SCHED_BREADTH_FIRST, se, si, after)
    after.synchronize()
    oc2 = torch.empty_like(oc1)
    om2 = torch.empty_like(om1)
    head.forward(x0, oc2, om2, dpi.DPI_SCHED_BREADTH_FIRST, se, si, after)
    after.synchronize()
    assert torch.equal(oc1, oc2) and torch.equal(om1, om2)
