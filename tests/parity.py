"""GPU-vs-oracle comparison helpers (test side only)."""
import numpy as np
import torch

import oracle
from cases import pooling_codes, sub_problem
from synth import configs, generate as G

TOL_F32_TABLES = 1e-5     # max componentwise relative error, fp32 tables
TOL_F16_TABLES = 2e-3     # fp16 tables, fp32 accumulation


def half_ulp_fp16(ref):
    """Half the binary16 spacing at |ref| (one output rounding)."""
    a = np.abs(ref).astype(np.float16)
    return 0.5 * np.spacing(a).astype(np.float64)


def check_outputs(y, ref, mag, table_f16, out_f16, exact=False, where=""):
    """Componentwise bound |y - ref| <= tol * mag (+ half an fp16 ulp for fp16
    output); elements whose magnitude is 0 must be exactly 0."""
    y = np.asarray(y, dtype=np.float64)
    assert y.shape == ref.shape, (y.shape, ref.shape)
    if exact:
        bad = np.argwhere(y != ref)
        assert bad.size == 0, f"{where}: {len(bad)} elements differ, first {bad[:3].tolist()}"
        return {"max_abs": 0.0}
    tol = TOL_F16_TABLES if table_f16 else TOL_F32_TABLES
    bound = tol * mag
    if out_f16:
        bound = bound + half_ulp_fp16(ref)
    err = np.abs(y - ref)
    zero = mag == 0
    assert np.all(y[zero] == 0), f"{where}: nonzero output where every term is zero"
    viol = err > bound
    if viol.any():
        i = np.argwhere(viol)[0]
        raise AssertionError(f"{where}: {viol.sum()} elements out of tolerance; first {tuple(i)}: "
                             f"y={y[tuple(i)]!r} ref={ref[tuple(i)]!r} mag={mag[tuple(i)]!r}")
    nz = mag > 0
    rel = float(np.max(err[nz] / mag[nz])) if nz.any() else 0.0
    return {"max_comp_rel": rel, "max_abs": float(err.max(initial=0.0))}


def oracle_ref(cfg, rotation=0, ranges=None, mapping="literal"):
    p = sub_problem(cfg, rotation, mapping=mapping, ranges=ranges)
    out, mag = oracle.lookup(p["dims"], p["tables"], p["ids"], p["offsets"], p["pooling"], p["B"])
    return p, out, mag


def gpu_tables(cfg, device="cuda"):
    return [G.make_table(cfg, t, device) for t in range(cfg.num_tables)]


def out_torch_dtype(cfg):
    return torch.float16 if cfg.out_dtype == configs.F16 else torch.float32


def plan_args(cfg):
    dims = [cfg.dim(t) for t in range(cfg.num_tables)]
    dtypes = [1 if cfg.dtype == configs.F16 else 0] * cfg.num_tables
    out_dtype = 1 if cfg.out_dtype == configs.F16 else 0
    return dims, dtypes, out_dtype


def default_waves(cfg, total_ids):
    """The library's documented default: max(min(16 * CUs, max(ceil(T*B/8),
    min(ceil(ids/32) + T*B, 8*T))), ceil((ids + T*B) / 2048), 1)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    T, B = cfg.num_tables, cfg.batch
    fill = min(16 * cus, max(-(-(T * B) // 8), min(-(-total_ids // 32) + T * B, 8 * T)))
    return max(fill, -(-(total_ids + T * B) // 2048), 1)


__all__ = ["check_outputs", "oracle_ref", "gpu_tables", "out_torch_dtype", "plan_args", "default_waves",
           "pooling_codes"]
