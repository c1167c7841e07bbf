"""CPU oracle for the fused multi-table lookup -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package.  It wraps ``liboracle.so`` (plain C, fp64, see oracle.c) with
numpy arrays and shares nothing with the GPU library.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

from .build import LIB, build

OK, BAD_ARG, BAD_OFFSETS, BAD_ID = 0, 1, 5, 6
FLAG_EXACT_SPLIT = 1 << 1

_libs = {}


def _load(path: Optional[str] = None):
    path = path or LIB
    if path not in _libs:
        if path == LIB and not os.path.exists(LIB):
            build()
        lib = ctypes.CDLL(path)
        p = ctypes.c_void_p
        lib.oracle_lookup.argtypes = [ctypes.c_int32, ctypes.c_int64, p, p, p, p, p, p, p, p, p,
                                      ctypes.c_int32]
        lib.oracle_lookup.restype = ctypes.c_int
        lib.oracle_plan.argtypes = [ctypes.c_int32, ctypes.c_int64, p, p, ctypes.c_int32, p,
                                    ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                    ctypes.c_uint32, p, p, p, p, p, p]
        lib.oracle_plan.restype = ctypes.c_int
        lib.oracle_plan_waves.argtypes = [ctypes.c_int64, p, ctypes.c_int64, p, p, p, p, p, p]
        lib.oracle_plan_waves.restype = ctypes.c_int
        lib.oracle_fm_second_order.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                               ctypes.c_int32, p, p, p]
        lib.oracle_fm_second_order.restype = ctypes.c_int
        _libs[path] = lib
    return _libs[path]


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle status {code}")
        self.code = code


def lookup(dims: Sequence[int], tables: Sequence[np.ndarray], ids: np.ndarray,
           offsets: Optional[np.ndarray], pooling: Optional[Sequence[int]], batch: int,
           with_mag: bool = True, nthreads: int = 0, lib_path: Optional[str] = None):
    """Pooled [batch, sum(dims)] fp64 result (and its magnitude bound)."""
    lib = _load(lib_path)
    T = len(dims)
    tabs = [np.ascontiguousarray(t) for t in tables]
    dtypes = np.array([1 if t.dtype == np.float16 else 0 for t in tabs], dtype=np.int32)
    for t in tabs:
        if t.dtype not in (np.float16, np.float32):
            raise TypeError(t.dtype)
    dims_a = np.ascontiguousarray(dims, dtype=np.int32)
    rows = np.array([t.shape[0] for t in tabs], dtype=np.int64)
    ptrs = (ctypes.c_void_p * T)(*[t.ctypes.data for t in tabs])
    ids_a = np.ascontiguousarray(ids, dtype=np.int32)
    off_a = None if offsets is None else np.ascontiguousarray(offsets, dtype=np.int32)
    pool = None if pooling is None else np.ascontiguousarray(pooling, dtype=np.int32)
    total_d = int(dims_a.sum())
    out = np.empty((batch, total_d), dtype=np.float64)
    mag = np.empty_like(out) if with_mag else None
    st = lib.oracle_lookup(T, batch, _ptr(rows), _ptr(dims_a), _ptr(dtypes),
                           ctypes.cast(ptrs, ctypes.c_void_p), _ptr(ids_a), _ptr(off_a), _ptr(pool),
                           _ptr(out), _ptr(mag), nthreads)
    if st != OK:
        raise OracleError(st)
    return (out, mag) if with_mag else out


def plan(dims: Sequence[int], dtypes: Sequence[int], out_dtype: int, offsets: Optional[np.ndarray],
         batch: int, total_ids: int, chunk_rows: int, item_cost_k: int, waves_requested: int,
         flags: int = 0, lib_path: Optional[str] = None):
    """Integer work plan; returns a dict of int64 arrays."""
    lib = _load(lib_path)
    T = len(dims)
    dims_a = np.ascontiguousarray(dims, dtype=np.int32)
    dt_a = np.ascontiguousarray(dtypes, dtype=np.int32)
    off_a = None if offsets is None else np.ascontiguousarray(offsets, dtype=np.int32)
    hdr = np.zeros(16, dtype=np.int64)
    col = np.zeros(T + 1, dtype=np.int64)
    idb = np.zeros(T + 1, dtype=np.int64)
    bib = np.zeros(T * batch + 1, dtype=np.int64)
    bcb = np.zeros(T * batch + 1, dtype=np.int64)
    wib = np.zeros(waves_requested + 1, dtype=np.int64)
    st = lib.oracle_plan(T, batch, _ptr(dims_a), _ptr(dt_a), out_dtype, _ptr(off_a), total_ids,
                         chunk_rows, item_cost_k, waves_requested, flags, _ptr(hdr), _ptr(col),
                         _ptr(idb), _ptr(bib), _ptr(bcb), _ptr(wib))
    if st != OK:
        raise OracleError(st)
    W = int(hdr[3])
    wib = np.ascontiguousarray(wib[: W + 1])
    res = {"header": hdr, "col_base": col, "id_base": idb, "bag_item_base": bib,
           "bag_cost_base": bcb, "wave_item_begin": wib}
    res.update(plan_waves(bib, wib, lib_path=lib_path))
    return res


def plan_waves(bag_item_base: np.ndarray, wave_item_begin: np.ndarray, lib_path: Optional[str] = None):
    """The per-wave arrays a lookup reads of a plan (closed forms of the wave starts
    and the bags' first items): wave_bag, wave_bag_base [W+1]; head_first,
    split_pieces, split_last [W] (int32)."""
    lib = _load(lib_path)
    bib = np.ascontiguousarray(bag_item_base, dtype=np.int64)
    wib = np.ascontiguousarray(wave_item_begin, dtype=np.int64)
    TB, W = len(bib) - 1, len(wib) - 1
    wb = np.zeros(W + 1, np.int64)
    wbb = np.zeros(W + 1, np.int64)
    hf = np.zeros(max(W, 1), np.int32)
    sp = np.zeros(max(W, 1), np.int32)
    sl = np.zeros(max(W, 1), np.int32)
    st = lib.oracle_plan_waves(TB, _ptr(bib), W, _ptr(wib), _ptr(wb), _ptr(wbb), _ptr(hf), _ptr(sp), _ptr(sl))
    if st != OK:
        raise OracleError(st)
    return {"wave_bag": wb, "wave_bag_base": wbb, "head_first": hf[:W], "split_pieces": sp[:W],
            "split_last": sl[:W]}


def fm_second_order(emb: np.ndarray, num_fields: int, dim: int, with_mag: bool = True,
                    lib_path: Optional[str] = None):
    """Second-order FM term per sample of a [batch, row_stride] fp16/fp32 block whose
    first num_fields * dim columns hold the fields; fp64 [batch] (and its magnitude)."""
    lib = _load(lib_path)
    e = np.ascontiguousarray(emb)
    if e.dtype not in (np.float16, np.float32) or e.ndim != 2:
        raise TypeError(e.dtype)
    B = e.shape[0]
    out = np.empty(B, dtype=np.float64)
    mag = np.empty(B, dtype=np.float64) if with_mag else None
    st = lib.oracle_fm_second_order(B, num_fields, dim, e.shape[1], 1 if e.dtype == np.float16 else 0,
                                    _ptr(e), _ptr(out), _ptr(mag))
    if st != OK:
        raise OracleError(st)
    return (out, mag) if with_mag else out


def stage_onehot(x: np.ndarray, num_fields: int) -> np.ndarray:
    """Field-major int32 ids from a sample-major feature matrix (the transpose of
    Algorithm 1's id matrix, §IV-B), as the input consolidation of the paper's
    breakdown (§V) produces them: ids[t * B + b] = x[b][t] when that value is an
    integer in [0, 2^31), else -1."""
    v = np.asarray(x)[:, :num_fields]
    if v.dtype.kind == "f":
        w = v.astype(np.float64)
        with np.errstate(invalid="ignore"):
            ok = np.isfinite(w) & (w >= 0) & (w < 2.0 ** 31) & (w == np.trunc(w))
        ints = np.where(ok, w, -1).astype(np.int64)
    else:
        w = v.astype(np.int64)
        ok = (w >= 0) & (w < 2 ** 31)
        ints = np.where(ok, w, -1)
    return np.ascontiguousarray(ints.T).reshape(-1).astype(np.int32)


def breadth_first_order(n_explicit: int, n_implicit: int):
    """Launch queue of Algorithm 2 (§IV-E): the two interaction modules' operators
    interleaved one by one, starting with the module that has more operators (the
    explicit one on a tie), the longer module's remaining operators at the end.
    Entries are ("E", i) for explicit operator i and ("I", j) for implicit operator j."""
    if n_implicit > n_explicit:
        first, second, n_first, n_second = "I", "E", n_implicit, n_explicit
    else:
        first, second, n_first, n_second = "E", "I", n_explicit, n_implicit
    q = []
    for i in range(n_second):
        q.append((first, i))
        q.append((second, i))
    for j in range(n_second, n_first):
        q.append((first, j))
    return q


def dcn_forward(x0: np.ndarray, cross_w, cross_b, mlp_w, mlp_b):
    """The interaction modules over the pooled block x0 [B, d], in fp64:
    explicit (a DCNv2 cross network, §IV-D): x_{l+1} = x0 * (x_l W_l^T + b_l) + x_l;
    implicit (an MLP): h_{l+1} = max(0, h_l V_l^T + c_l).
    Returns (x_L, h_M, mag_x, mag_h): the magnitudes are the same networks run on
    absolute values without the ReLU, the scale of the error bounds."""
    x0 = np.asarray(x0, np.float64)
    ax0 = np.abs(x0)
    x, ax = x0.copy(), ax0.copy()
    for W, b in zip(cross_w, cross_b):
        W, b = np.asarray(W, np.float64), np.asarray(b, np.float64)
        x = x0 * (x @ W.T + b) + x
        ax = ax0 * (ax @ np.abs(W).T + np.abs(b)) + ax
    h, ah = x0.copy(), ax0.copy()
    for V, c in zip(mlp_w, mlp_b):
        V, c = np.asarray(V, np.float64), np.asarray(c, np.float64)
        h = np.maximum(0.0, h @ V.T + c)
        ah = ah @ np.abs(V).T + np.abs(c)
    return x, h, ax, ah


def stage_csr(packed: np.ndarray, num_fields: int, batch: int, total_ids: int):
    """Multi-hot input consolidation (§V breakdown): one packed host array holding
    every field's offsets ([T][B+1], local per field) followed by the fields'
    concatenated ids, as a loader produces them; returns the int32 offsets and ids
    the plan and lookup take.  A value that is not an integer in [0, 2^31) becomes -1."""
    v = np.asarray(packed)
    n_off = num_fields * (batch + 1)
    if v.dtype.kind == "f":
        w = v.astype(np.float64)
        with np.errstate(invalid="ignore"):
            ok = np.isfinite(w) & (w >= 0) & (w < 2.0 ** 31) & (w == np.trunc(w))
        ints = np.where(ok, w, -1).astype(np.int64)
    else:
        w = v.astype(np.int64)
        ints = np.where((w >= 0) & (w < 2 ** 31), w, -1)
    return (ints[:n_off].astype(np.int32).reshape(num_fields, batch + 1),
            ints[n_off:n_off + total_ids].astype(np.int32))
