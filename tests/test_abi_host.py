"""The C ABI library loads, exports every declared symbol and validates its
host-visible arguments before touching the GPU (runs without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2606_21101_amd import dpi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "dpi.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dpi_[a-z_]+)\s*\((?!\s*\*)", text)))


def test_exports_every_declared_symbol():
    lib = dpi.load()
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_strings():
    assert dpi.dpi_abi_version() == 1
    for s in range(8):
        assert dpi.dpi_status_str(s)
    assert "unknown" in dpi.dpi_status_str(99)


def _gpu_present():
    import torch
    return torch.cuda.device_count() > 0


def _meta(dims=(16, 16), dtypes=(0, 0), rows=(10, 10)):
    return dpi.make_meta(rows, dims, dtypes)


def _plan(meta, T=None, offsets=None, B=4, total=None, opts=None, ws=0x10000, ws_bytes=1 << 30):
    lib = dpi.load()
    T = len(meta) if T is None else T
    total = T * B if total is None else total
    out = ctypes.c_void_p()
    o = opts if opts is not None else dpi.make_opts(num_waves=64)
    return lib.dpi_plan(meta, T, offsets, B, total, ctypes.byref(o), ws, ws_bytes, None, ctypes.byref(out))


def test_plan_rejects_bad_arguments():
    lib = dpi.load()
    m = _meta()
    assert lib.dpi_plan(m, 2, None, 4, 8, None, 0x10000, 1 << 30, None, None) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(None, T=2) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(m, T=0) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(_meta(dims=[4] * 257, dtypes=[0] * 257, rows=[1] * 257)) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(m, B=-1) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(m, total=7) == dpi.DPI_ERR_INVALID_ARG          # one-hot needs T*B ids
    assert _plan(_meta(dtypes=(0, 2))) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(_meta(dims=(16, 0))) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(_meta(rows=(10, -1))) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(m, opts=dpi.make_opts(num_waves=64, out_dtype=3)) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(m, opts=dpi.make_opts(num_waves=64, flags=1 << 9)) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(m, opts=dpi.make_opts(chunk_rows=-1, num_waves=64)) == dpi.DPI_ERR_INVALID_ARG
    assert "one-hot" in dpi.dpi_last_error() or dpi.dpi_last_error()


def test_plan_rejects_unsupported_and_misaligned():
    assert _plan(_meta(dims=(3, 16), dtypes=(1, 0))) == dpi.DPI_ERR_UNSUPPORTED   # 6-byte rows
    assert _plan(_meta(dims=(70000, 16))) == dpi.DPI_ERR_UNSUPPORTED
    assert _plan(_meta(), ws=0x10008) == dpi.DPI_ERR_MISALIGNED
    assert _plan(_meta(), offsets=0x10002, total=3) == dpi.DPI_ERR_MISALIGNED
    assert _plan(_meta(), ws=None) == dpi.DPI_ERR_INVALID_ARG
    assert _plan(_meta(), ws_bytes=100) == dpi.DPI_ERR_WORKSPACE_TOO_SMALL
    assert "need" in dpi.dpi_last_error()


def test_workspace_size_query():
    o = dpi.make_opts(num_waves=100)
    a = dpi.dpi_plan_workspace_bytes(26, 16384, 4_000_000, 64, o)
    b = dpi.dpi_plan_workspace_bytes(26, 16384, 4_000_000, 128, o)
    assert 0 < a < b
    assert dpi.dpi_plan_workspace_bytes(0, 1, 1, 16, o) == 0
    assert dpi.dpi_plan_workspace_bytes(1, -1, 1, 16, o) == 0
    assert dpi.dpi_plan_workspace_bytes(1, 1, 1, 0, o) == 0


def test_lookup_rejects_null_plan_and_destroy_null():
    lib = dpi.load()
    ptrs = (ctypes.c_void_p * 1)(0x10000)
    assert lib.dpi_lookup(None, ptrs, 0x10000, None, None, 0x10000, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_plan_sync_status(None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_plan_export(None, None, None, None, None, None, None) == dpi.DPI_ERR_INVALID_ARG
    lib.dpi_plan_destroy(None)


def default_waves_rule(T, B, ids, cus=256):
    by_work = -(-(ids + T * B) // 2048)
    fill = min(16 * cus, max(-(-(T * B) // 8), min(-(-ids // 32) + T * B, 8 * T)))
    return max(fill, by_work, 1)


def test_default_waves_formula():
    # on a host without a GPU the CU count falls back to 256
    assert dpi.dpi_default_waves(100, 65536, 176_805_878) == -(-(176_805_878 + 100 * 65536) // 2048)
    assert dpi.dpi_default_waves(26, 16384, 4_260_852) == 16 * 256
    for T, B, ids, want in ((39, 1, 552, 57), (39, 16, 8588, 312), (39, 128, 67979, 624), (39, 512, 272316, 2496),
                            (39, 4096, 2173692, 4096), (8, 256, 2048, 256), (1, 0, 0, 1)):
        assert dpi.dpi_default_waves(T, B, ids) == want == default_waves_rule(T, B, ids)


def test_fm_host_validation():
    lib = dpi.load()
    vp = 0x10000
    assert lib.dpi_fm_second_order(None, dpi.DPI_F32, 0, 3, 4, 12, None, None) == dpi.DPI_OK
    assert lib.dpi_fm_second_order(vp, dpi.DPI_F32, -1, 3, 4, 12, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_fm_second_order(vp, dpi.DPI_F32, 2, 0, 4, 12, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_fm_second_order(vp, dpi.DPI_F32, 2, 3, 4, 11, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_fm_second_order(vp, 7, 2, 3, 4, 12, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_fm_second_order(vp, dpi.DPI_F32, 2, 3, 70000, 1 << 20, vp, None) == dpi.DPI_ERR_UNSUPPORTED
    assert lib.dpi_fm_second_order(vp + 2, dpi.DPI_F32, 2, 3, 4, 12, vp, None) == dpi.DPI_ERR_MISALIGNED
    assert lib.dpi_fm_second_order(vp, dpi.DPI_F32, 2, 3, 4, 12, vp + 2, None) == dpi.DPI_ERR_MISALIGNED


def test_stage_host_validation():
    lib = dpi.load()
    vp = 0x10000
    assert lib.dpi_stage_onehot(None, dpi.DPI_X_F32, 0, 3, 4, None, 0, None, None) == dpi.DPI_OK
    assert lib.dpi_stage_onehot(vp, dpi.DPI_X_F32, -1, 3, 4, vp, 1 << 20, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_stage_onehot(vp, dpi.DPI_X_F32, 2, 5, 4, vp, 1 << 20, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_stage_onehot(vp, 9, 2, 3, 4, vp, 1 << 20, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_stage_onehot(vp, dpi.DPI_X_I64, 2, 3, 4, vp, 63, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_stage_onehot(vp, dpi.DPI_X_F32, 2, 3, 4, vp + 4, 1 << 20, vp, None) == dpi.DPI_ERR_MISALIGNED
    assert lib.dpi_stage_onehot(vp, dpi.DPI_X_F32, 2, 3, 4, vp, 1 << 20, vp + 2, None) == dpi.DPI_ERR_MISALIGNED


def test_breadth_first_order_matches_oracle():
    import oracle
    for ne in range(6):
        for ni in range(6):
            got = dpi.dpi_breadth_first_order(ne, ni)
            want = [i if k == "E" else -(i + 1) for k, i in oracle.breadth_first_order(ne, ni)]
            assert got == want


def test_scheduler_host_validation():
    lib = dpi.load()
    none = (dpi.dpi_op * 1)()
    assert lib.dpi_breadth_first_order(-1, 2, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_breadth_first_order(1, 2, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_launch_two_streams(none, 1, none, 1, 0, None, None, None) == dpi.DPI_ERR_INVALID_ARG  # no launch fn
    assert lib.dpi_launch_two_streams(None, 1, None, 0, 0, None, None, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_launch_two_streams(none, 0, none, 0, 9, None, None, None) == dpi.DPI_ERR_INVALID_ARG
    d = dpi.dpi_dcn_desc()
    assert lib.dpi_dcn_workspace_bytes(ctypes.byref(d)) == 0          # batch 0, no layers
    out = ctypes.c_void_p()
    assert lib.dpi_dcn_create(ctypes.byref(d), None, 0, ctypes.byref(out)) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_dcn_forward(None, None, None, None, 0, None, None, None, None) == dpi.DPI_ERR_INVALID_ARG


def test_stage_csr_host_validation():
    lib = dpi.load()
    vp = 0x10000
    assert lib.dpi_stage_csr(vp, dpi.DPI_X_I64, 0, 2, 4, vp, 1 << 20, vp, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_stage_csr(vp, dpi.DPI_X_I64, 2, -1, 4, vp, 1 << 20, vp, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_stage_csr(vp, 5, 2, 2, 4, vp, 1 << 20, vp, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_stage_csr(None, dpi.DPI_X_I64, 2, 2, 4, vp, 1 << 20, vp, vp, None) == dpi.DPI_ERR_INVALID_ARG
    assert lib.dpi_stage_csr(vp, dpi.DPI_X_I64, 2, 2, 4, vp, 79, vp, vp, None) == dpi.DPI_ERR_INVALID_ARG  # 10 * 8 bytes
    assert lib.dpi_stage_csr(vp, dpi.DPI_X_I64, 2, 2, 4, vp + 8, 1 << 20, vp, vp, None) == dpi.DPI_ERR_MISALIGNED
    assert lib.dpi_stage_csr(vp + 4, dpi.DPI_X_I64, 2, 2, 4, vp, 1 << 20, vp, vp, None) == dpi.DPI_ERR_MISALIGNED


def test_binding_constants_mirror_the_header():
    text = open(os.path.join(ROOT, "include", "dpi.h")).read()
    for name, value in re.findall(r"#define (DPI_[A-Z_]+)\s+(\d+)", text):
        assert getattr(dpi, name) == int(value), name
    enums = dict(re.findall(r"\b(DPI_[A-Z0-9_]+) = (\d+)\b", text))
    shifts = dict(re.findall(r"\b(DPI_FLAG_[A-Z_]+) = 1u << (\d+)", text))
    for name, value in enums.items():
        assert getattr(dpi, name) == int(value), name
    for name, bit in shifts.items():
        assert getattr(dpi, name) == 1 << int(bit), name


def test_one_launch_plans_enqueue_nothing():
    """Bag-by-bag and one-hot batches of at most 64 fields (and 1024 bags per
    field with offsets) plan on the host alone: dpi_plan succeeds with no
    device present, while a plan that needs its planning launch reports the
    HIP error of that launch."""
    if _gpu_present():
        pytest.skip("needs a host without a GPU")
    lib = dpi.load()
    m = _meta()
    for offsets, B, total, opts in ((0x10000, 4, 8, dpi.make_opts()), (None, 4, 8, dpi.make_opts()),
                                    (0x10000, 1024, 3000, dpi.make_opts()), (None, 5000, 10000, dpi.make_opts())):
        out = ctypes.c_void_p()
        assert lib.dpi_plan(m, 2, offsets, B, total, ctypes.byref(opts), 0x20000, 1 << 30, None,
                            ctypes.byref(out)) == dpi.DPI_OK, dpi.dpi_last_error()
        lib.dpi_plan_destroy(out)
    for offsets, B, total, opts in ((0x10000, 4, 8, dpi.make_opts(num_waves=64)),     # explicit wave count
                                    (0x10000, 1025, 3000, dpi.make_opts())):           # more than 1024 bags
        out = ctypes.c_void_p()
        assert lib.dpi_plan(m, 2, offsets, B, total, ctypes.byref(opts), 0x20000, 1 << 30, None,
                            ctypes.byref(out)) == dpi.DPI_ERR_HIP
    wide = _meta(dims=[16] * 65, dtypes=[0] * 65, rows=[10] * 65)
    out = ctypes.c_void_p()
    assert lib.dpi_plan(wide, 65, 0x10000, 4, 8, ctypes.byref(dpi.make_opts()), 0x20000, 1 << 30, None,
                        ctypes.byref(out)) == dpi.DPI_ERR_HIP                          # 65 fields


def test_lookup_csr_host_validation():
    lib = dpi.load()
    vp = 0x10000
    tabs = (ctypes.c_void_p * 2)(0x30000, 0x30000)
    assert lib.dpi_lookup_csr(None, vp, dpi.DPI_X_I64, 0x40000, 1 << 20, tabs, None, vp, vp, 0x50000,
                              None) == dpi.DPI_ERR_INVALID_ARG
    if _gpu_present():
        return
    out = ctypes.c_void_p()
    assert lib.dpi_plan(_meta(), 2, vp, 4, 8, ctypes.byref(dpi.make_opts()), 0x20000, 1 << 30, None,
                        ctypes.byref(out)) == dpi.DPI_OK
    args = dict(packed=vp, x=dpi.DPI_X_I64, staging=0x40000, sbytes=1 << 20, offsets=vp)

    def call(**kw):
        a = {**args, **kw}
        return lib.dpi_lookup_csr(out, a["packed"], a["x"], a["staging"], a["sbytes"], tabs, None, a["offsets"], vp,
                                  0x50000, None)
    assert call(offsets=vp + 4) == dpi.DPI_ERR_INVALID_ARG       # not the plan's offsets
    assert call(x=7) == dpi.DPI_ERR_INVALID_ARG
    assert call(sbytes=8 * 17) == dpi.DPI_ERR_INVALID_ARG        # 2 * 5 offsets + 8 ids = 18 elements
    assert call(staging=0x40008) == dpi.DPI_ERR_MISALIGNED
    assert call(packed=vp + 4) == dpi.DPI_ERR_MISALIGNED
    later = ctypes.c_void_p()
    assert lib.dpi_plan(_meta(), 2, vp, 4, 8, ctypes.byref(dpi.make_opts()), 0x20000, 1 << 30, None,
                        ctypes.byref(later)) == dpi.DPI_OK
    assert call() == dpi.DPI_ERR_INVALID_ARG and "later plan" in dpi.dpi_last_error()
    lib.dpi_plan_destroy(out)
    lib.dpi_plan_destroy(later)
