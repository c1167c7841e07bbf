"""Python binding of the C ABI in include/dpi.h (ctypes; argument marshalling only).

Every step of the lookup runs in libdpi.so's HIP kernels.  torch tensors are
accepted wherever the ABI takes device memory: only their data pointers are
passed.  There is no fallback: if the library is not built, loading fails.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

from .build import LIB

DPI_OK = 0
DPI_ERR_INVALID_ARG = 1
DPI_ERR_UNSUPPORTED = 2
DPI_ERR_MISALIGNED = 3
DPI_ERR_WORKSPACE_TOO_SMALL = 4
DPI_ERR_BAD_OFFSETS = 5
DPI_ERR_BAD_ID = 6
DPI_ERR_HIP = 7

DPI_F32 = 0
DPI_F16 = 1
DPI_X_F32 = 0
DPI_X_I64 = 1
DPI_X_I32 = 2
DPI_POOL_SUM = 0
DPI_POOL_MEAN = 1
DPI_FLAG_EXACT_SPLIT = 1 << 1
DPI_FLAG_LINEAR_BLOCKS = 1 << 2
DPI_FLAG_INPUT_FIRST = 1 << 3
DPI_SCHED_BREADTH_FIRST = 0
DPI_SCHED_DEPTH_FIRST = 1
DPI_SCHED_ONE_STREAM = 2
DPI_ABI_VERSION = 1
DPI_MAX_TABLES = 256
DPI_MAX_DIM = 65536
DPI_NOALLOC_SCRATCH_BYTES = 64 << 20
DPI_DEVSTAT_BAD_OFFSETS = 1
DPI_DEVSTAT_BAD_ID = 2


class dpi_table_meta(ctypes.Structure):
    _fields_ = [("num_rows", ctypes.c_int64), ("dim", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class dpi_plan_opts(ctypes.Structure):
    _fields_ = [("chunk_rows", ctypes.c_int32), ("item_cost_k", ctypes.c_int32), ("num_waves", ctypes.c_int64),
                ("out_dtype", ctypes.c_int32), ("flags", ctypes.c_uint32)]


DPI_OP_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p)


class dpi_op(ctypes.Structure):
    _fields_ = [("launch", DPI_OP_FN), ("ctx", ctypes.c_void_p)]


class dpi_dcn_desc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("dim", ctypes.c_int32), ("n_cross", ctypes.c_int32),
                ("n_mlp", ctypes.c_int32), ("mlp_dims", ctypes.POINTER(ctypes.c_int32)),
                ("cross_w", ctypes.POINTER(ctypes.c_void_p)), ("cross_b", ctypes.POINTER(ctypes.c_void_p)),
                ("mlp_w", ctypes.POINTER(ctypes.c_void_p)), ("mlp_b", ctypes.POINTER(ctypes.c_void_p))]


class DpiError(RuntimeError):
    def __init__(self, status: int, detail: str = ""):
        self.status = status
        super().__init__(f"{dpi_status_str(status)} ({status}): {detail}")


_lib = None


def load() -> ctypes.CDLL:
    """Load the in-tree libdpi.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB):
        raise ImportError(f"{LIB} is missing: build it with __graft_entry__.build() "
                          "(hipcc --offload-arch=gfx950); there is no CPU fallback")
    lib = ctypes.CDLL(LIB)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.dpi_abi_version.restype = ctypes.c_int
    lib.dpi_last_error.restype = ctypes.c_char_p
    lib.dpi_status_str.restype = ctypes.c_char_p
    lib.dpi_status_str.argtypes = [ctypes.c_int]
    lib.dpi_default_waves.restype = i64
    lib.dpi_default_waves.argtypes = [i32, i64, i64]
    lib.dpi_plan_workspace_bytes.restype = sz
    lib.dpi_plan_workspace_bytes.argtypes = [i32, i64, i64, i32, ctypes.POINTER(dpi_plan_opts)]
    lib.dpi_plan.restype = ctypes.c_int
    lib.dpi_plan.argtypes = [ctypes.POINTER(dpi_table_meta), i32, vp, i64, i64, ctypes.POINTER(dpi_plan_opts),
                             vp, sz, vp, ctypes.POINTER(vp)]
    lib.dpi_lookup.restype = ctypes.c_int
    lib.dpi_lookup.argtypes = [vp, ctypes.POINTER(vp), vp, vp, ctypes.POINTER(i32), vp, vp]
    lib.dpi_plan_sync_status.restype = ctypes.c_int
    lib.dpi_plan_sync_status.argtypes = [vp]
    p64 = ctypes.POINTER(i64)
    lib.dpi_plan_export.restype = ctypes.c_int
    lib.dpi_plan_export.argtypes = [vp, p64, p64, p64, p64, p64, p64]
    p32 = ctypes.POINTER(i32)
    lib.dpi_plan_export_waves.restype = ctypes.c_int
    lib.dpi_plan_export_waves.argtypes = [vp, p64, p64, p32, p32, p32, p32]
    lib.dpi_fm_second_order.restype = ctypes.c_int
    lib.dpi_fm_second_order.argtypes = [vp, i32, i64, i32, i32, i64, vp, vp]
    lib.dpi_stage_onehot.restype = ctypes.c_int
    lib.dpi_stage_onehot.argtypes = [vp, i32, i64, i32, i64, vp, sz, vp, vp]
    lib.dpi_stage_csr.restype = ctypes.c_int
    lib.dpi_stage_csr.argtypes = [vp, i32, i32, i64, i64, vp, sz, vp, vp, vp]
    lib.dpi_lookup_csr.restype = ctypes.c_int
    lib.dpi_lookup_csr.argtypes = [vp, vp, i32, vp, sz, ctypes.POINTER(vp), ctypes.POINTER(i32), vp, vp, vp, vp]
    lib.dpi_breadth_first_order.restype = ctypes.c_int
    lib.dpi_breadth_first_order.argtypes = [i32, i32, ctypes.POINTER(i32)]
    lib.dpi_launch_two_streams.restype = ctypes.c_int
    lib.dpi_launch_two_streams.argtypes = [ctypes.POINTER(dpi_op), i32, ctypes.POINTER(dpi_op), i32, i32, vp, vp, vp]
    lib.dpi_wall_clock_khz.restype = i64
    lib.dpi_wall_clock_khz.argtypes = []
    lib.dpi_dcn_workspace_bytes.restype = sz
    lib.dpi_dcn_workspace_bytes.argtypes = [ctypes.POINTER(dpi_dcn_desc)]
    lib.dpi_dcn_create.restype = ctypes.c_int
    lib.dpi_dcn_create.argtypes = [ctypes.POINTER(dpi_dcn_desc), vp, sz, ctypes.POINTER(vp)]
    lib.dpi_dcn_forward.restype = ctypes.c_int
    lib.dpi_dcn_forward.argtypes = [vp, vp, vp, vp, i32, vp, vp, vp, vp]
    lib.dpi_dcn_destroy.restype = None
    lib.dpi_dcn_destroy.argtypes = [vp]
    lib.dpi_lookup_noalloc.restype = ctypes.c_int
    lib.dpi_lookup_noalloc.argtypes = [ctypes.POINTER(dpi_table_meta), i32, ctypes.POINTER(vp), vp, vp, i64, i64,
                                       ctypes.POINTER(i32), ctypes.POINTER(dpi_plan_opts), vp, vp, vp]
    lib.dpi_plan_destroy.restype = None
    lib.dpi_plan_destroy.argtypes = [vp]
    _lib = lib
    return lib


def _ptr(x) -> Optional[int]:
    """Device (or host) address of a tensor, an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(stream) -> Optional[int]:
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def _check(status: int):
    if status != DPI_OK:
        raise DpiError(status, dpi_last_error())


def dpi_abi_version() -> int:
    return load().dpi_abi_version()


def dpi_last_error() -> str:
    return load().dpi_last_error().decode()


def dpi_status_str(status: int) -> str:
    return load().dpi_status_str(int(status)).decode()


def dpi_default_waves(num_tables: int, batch: int, total_ids: int) -> int:
    return int(load().dpi_default_waves(num_tables, batch, total_ids))


def make_opts(chunk_rows: int = 0, item_cost_k: int = 0, num_waves: int = 0, out_dtype: int = DPI_F32,
              flags: int = 0) -> dpi_plan_opts:
    return dpi_plan_opts(chunk_rows, item_cost_k, num_waves, out_dtype, flags)


def make_meta(num_rows: Sequence[int], dims: Sequence[int], dtypes: Sequence[int]):
    T = len(dims)
    arr = (dpi_table_meta * T)()
    for t in range(T):
        arr[t] = dpi_table_meta(int(num_rows[t]), int(dims[t]), int(dtypes[t]))
    return arr


def dpi_plan_workspace_bytes(num_tables: int, batch: int, total_ids: int, max_dim: int,
                             opts: Optional[dpi_plan_opts] = None) -> int:
    o = ctypes.byref(opts) if opts is not None else None
    return int(load().dpi_plan_workspace_bytes(num_tables, batch, total_ids, max_dim, o))


@dataclass
class Plan:
    """Handle of a device plan; keeps the borrowed buffers alive.  A workspace
    holds one plan at a time: planning into it again supersedes the plan before,
    which the library then refuses for lookups, status queries and exports."""
    handle: int
    num_tables: int
    batch: int
    keep: tuple

    def __del__(self):
        if self.handle and _lib is not None:
            _lib.dpi_plan_destroy(ctypes.c_void_p(self.handle))
            self.handle = 0


def dpi_plan(table_meta, offsets, batch: int, total_ids: int, opts: Optional[dpi_plan_opts], workspace,
             workspace_bytes: Optional[int] = None, stream=None) -> Plan:
    lib = load()
    T = len(table_meta)
    if workspace_bytes is None:
        workspace_bytes = int(workspace.numel() * workspace.element_size())
    out = ctypes.c_void_p()
    st = lib.dpi_plan(table_meta, T, _ptr(offsets), batch, total_ids,
                      ctypes.byref(opts) if opts is not None else None, _ptr(workspace), workspace_bytes,
                      _stream(stream), ctypes.byref(out))
    _check(st)
    return Plan(out.value, T, batch, (workspace, offsets, table_meta))


def table_array(tables) -> ctypes.Array:
    """Host array of the tables' device pointers, as dpi_lookup takes it (build it
    once and pass it to every lookup over the same tables)."""
    return (ctypes.c_void_p * len(tables))(*[_ptr(t) for t in tables])


def pooling_array(pooling: Sequence[int]) -> ctypes.Array:
    return (ctypes.c_int32 * len(pooling))(*[int(p) for p in pooling])


def dpi_lookup(plan: Plan, tables, ids, offsets, pooling: Optional[Sequence[int]], out, stream=None) -> None:
    """tables / pooling: sequences, or the arrays table_array / pooling_array built."""
    lib = load()
    T = plan.num_tables
    ptrs = tables if isinstance(tables, ctypes.Array) else table_array(tables)
    pool = pooling if (pooling is None or isinstance(pooling, ctypes.Array)) else pooling_array(pooling)
    if len(ptrs) != T or (pool is not None and len(pool) != T):
        raise DpiError(DPI_ERR_INVALID_ARG, "tables / pooling must have one entry per field")
    st = lib.dpi_lookup(ctypes.c_void_p(plan.handle), ptrs, _ptr(ids), _ptr(offsets), pool, _ptr(out),
                        _stream(stream))
    _check(st)


def dpi_lookup_noalloc(table_meta, tables, ids, offsets, batch: int, total_ids: int,
                       pooling: Optional[Sequence[int]], opts: Optional[dpi_plan_opts], out, device_status=None,
                       stream=None) -> None:
    """dpi_plan + dpi_lookup in one call with the library's fixed device scratch as the
    workspace (no allocation; see include/dpi.h).  tables / pooling: sequences, or the
    arrays table_array / pooling_array built."""
    lib = load()
    T = len(table_meta)
    ptrs = tables if isinstance(tables, ctypes.Array) else table_array(tables)
    pool = pooling if (pooling is None or isinstance(pooling, ctypes.Array)) else pooling_array(pooling)
    if len(ptrs) != T or (pool is not None and len(pool) != T):
        raise DpiError(DPI_ERR_INVALID_ARG, "tables / pooling must have one entry per field")
    _check(lib.dpi_lookup_noalloc(table_meta, T, ptrs, _ptr(ids), _ptr(offsets), batch, total_ids, pool,
                                  ctypes.byref(opts) if opts is not None else None, _ptr(out), _ptr(device_status),
                                  _stream(stream)))


def dpi_plan_sync_status(plan: Plan) -> int:
    """Device-detected status (an int dpi_status; does not raise)."""
    return int(load().dpi_plan_sync_status(ctypes.c_void_p(plan.handle)))


def dpi_plan_export(plan: Plan) -> dict:
    lib = load()
    hdr = np.zeros(16, dtype=np.int64)
    p64 = ctypes.POINTER(ctypes.c_int64)
    _check(lib.dpi_plan_export(ctypes.c_void_p(plan.handle), hdr.ctypes.data_as(p64), None, None, None, None, None))
    T, B, W = int(hdr[1]), int(hdr[2]), int(hdr[3])
    col = np.zeros(T + 1, np.int64)
    idb = np.zeros(T + 1, np.int64)
    bib = np.zeros(T * B + 1, np.int64)
    bcb = np.zeros(T * B + 1, np.int64)
    wib = np.zeros(W + 1, np.int64)
    _check(lib.dpi_plan_export(ctypes.c_void_p(plan.handle), hdr.ctypes.data_as(p64), col.ctypes.data_as(p64),
                               idb.ctypes.data_as(p64), bib.ctypes.data_as(p64), bcb.ctypes.data_as(p64),
                               wib.ctypes.data_as(p64)))
    return {"header": hdr, "col_base": col, "id_base": idb, "bag_item_base": bib, "bag_cost_base": bcb,
            "wave_item_begin": wib}


def dpi_plan_export_waves(plan: Plan) -> dict:
    """What a lookup reads of the plan besides the wave starts; "source" is 1 when
    these are the arrays the planning launch wrote (see include/dpi.h)."""
    lib = load()
    hdr = np.zeros(16, dtype=np.int64)
    p64 = ctypes.POINTER(ctypes.c_int64)
    p32 = ctypes.POINTER(ctypes.c_int32)
    _check(lib.dpi_plan_export(ctypes.c_void_p(plan.handle), hdr.ctypes.data_as(p64), None, None, None, None, None))
    W = int(hdr[3])
    wb = np.zeros(W + 1, np.int64)
    wbb = np.zeros(W + 1, np.int64)
    hf = np.zeros(max(W, 1), np.int32)
    sp = np.zeros(max(W, 1), np.int32)
    sl = np.zeros(max(W, 1), np.int32)
    src = ctypes.c_int32(-1)
    _check(lib.dpi_plan_export_waves(ctypes.c_void_p(plan.handle), wb.ctypes.data_as(p64), wbb.ctypes.data_as(p64),
                                     hf.ctypes.data_as(p32), sp.ctypes.data_as(p32), sl.ctypes.data_as(p32),
                                     ctypes.byref(src)))
    return {"wave_bag": wb, "wave_bag_base": wbb, "head_first": hf[:W], "split_pieces": sp[:W],
            "split_last": sl[:W], "source": int(src.value)}


def dpi_fm_second_order(emb, emb_dtype: int, batch: int, num_fields: int, dim: int, row_stride: int, out,
                        stream=None) -> None:
    """Second-order FM term per sample of a [batch, row_stride] block (fp32 out[batch])."""
    _check(load().dpi_fm_second_order(_ptr(emb), emb_dtype, batch, num_fields, dim, row_stride, _ptr(out),
                                      _stream(stream)))


def dpi_stage_onehot(x, x_dtype: int, batch: int, num_fields: int, row_stride: int, staging, ids,
                     staging_bytes: Optional[int] = None, stream=None) -> None:
    """One host-to-device copy of a sample-major feature matrix and one conversion kernel
    into field-major int32 ids (x: host memory, ideally pinned)."""
    if staging_bytes is None:
        staging_bytes = int(staging.numel() * staging.element_size())
    _check(load().dpi_stage_onehot(_ptr(x), x_dtype, batch, num_fields, row_stride, _ptr(staging),
                                   staging_bytes, _ptr(ids), _stream(stream)))


def dpi_breadth_first_order(n_explicit: int, n_implicit: int) -> list:
    """Algorithm 2's queue: i for explicit operator i, -(j + 1) for implicit operator j."""
    n = n_explicit + n_implicit
    arr = (ctypes.c_int32 * max(1, n))()
    _check(load().dpi_breadth_first_order(n_explicit, n_implicit, arr))
    return [int(arr[k]) for k in range(n)]


def dpi_launch_two_streams(explicit_ops, implicit_ops, mode: int, stream_explicit, stream_implicit, after) -> None:
    """explicit_ops / implicit_ops: sequences of dpi_op."""
    ne, ni = len(explicit_ops), len(implicit_ops)
    ea = (dpi_op * max(1, ne))(*explicit_ops)
    ia = (dpi_op * max(1, ni))(*implicit_ops)
    _check(load().dpi_launch_two_streams(ea, ne, ia, ni, mode, _stream(stream_explicit), _stream(stream_implicit),
                                         _stream(after)))


def dpi_wall_clock_khz() -> int:
    return int(load().dpi_wall_clock_khz())


class DcnHead:
    """dpi_dcn_t over torch fp32 weights (kept alive here): cross network + MLP."""

    def __init__(self, batch: int, dim: int, cross_w, cross_b, mlp_w, mlp_b, device=None):
        import torch
        lib = load()
        self.keep = [list(cross_w), list(cross_b), list(mlp_w), list(mlp_b)]
        self.mlp_dims = [int(w.shape[0]) for w in mlp_w]
        dims = (ctypes.c_int32 * len(self.mlp_dims))(*self.mlp_dims)
        ptrs = [(ctypes.c_void_p * max(1, len(v)))(*[_ptr(t) for t in v]) for v in self.keep]
        self._c = (dims, ptrs)
        self.desc = dpi_dcn_desc(batch, dim, len(cross_w), len(mlp_w), dims, ptrs[0], ptrs[1], ptrs[2], ptrs[3])
        need = int(lib.dpi_dcn_workspace_bytes(ctypes.byref(self.desc)))
        if need == 0:
            raise DpiError(DPI_ERR_INVALID_ARG, "dpi_dcn_workspace_bytes failed")
        dev = device if device is not None else cross_w[0].device
        self.ws = torch.empty(need + 256, dtype=torch.uint8, device=dev)
        base = _ptr(self.ws)
        off = (-base) % 256
        h = ctypes.c_void_p()
        _check(lib.dpi_dcn_create(ctypes.byref(self.desc), base + off, need, ctypes.byref(h)))
        self.handle = h.value
        self.batch, self.dim = batch, dim

    def forward(self, x0, out_cross, out_mlp, mode: int = DPI_SCHED_BREADTH_FIRST, stream_explicit=None,
                stream_implicit=None, after=None, marks=None) -> None:
        _check(load().dpi_dcn_forward(ctypes.c_void_p(self.handle), _ptr(x0), _ptr(out_cross), _ptr(out_mlp), mode,
                                      _stream(stream_explicit), _stream(stream_implicit), _stream(after),
                                      _ptr(marks)))

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.dpi_dcn_destroy(ctypes.c_void_p(self.handle))
            self.handle = None


def dpi_stage_csr(packed, x_dtype: int, num_fields: int, batch: int, total_ids: int, staging, offsets, ids,
                  staging_bytes: Optional[int] = None, stream=None) -> None:
    """One host-to-device copy of [all fields' offsets | all ids] and one conversion
    kernel into the int32 offsets and ids of dpi_plan / dpi_lookup."""
    if staging_bytes is None:
        staging_bytes = int(staging.numel() * staging.element_size())
    _check(load().dpi_stage_csr(_ptr(packed), x_dtype, num_fields, batch, total_ids, _ptr(staging), staging_bytes,
                                _ptr(offsets), _ptr(ids), _stream(stream)))


def dpi_lookup_csr(plan: Plan, packed, x_dtype: int, staging, tables, pooling: Optional[Sequence[int]], offsets, ids,
                   out, staging_bytes: Optional[int] = None, stream=None) -> None:
    """One copy of the packed host CSR into `staging` and one lookup kernel that
    converts it as it reads it (writing the int32 offsets and ids) and pools; for
    plans whose lookups take one launch (see include/dpi.h)."""
    lib = load()
    T = plan.num_tables
    if staging_bytes is None:
        staging_bytes = int(staging.numel() * staging.element_size())
    ptrs = tables if isinstance(tables, ctypes.Array) else table_array(tables)
    pool = pooling if (pooling is None or isinstance(pooling, ctypes.Array)) else pooling_array(pooling)
    if len(ptrs) != T or (pool is not None and len(pool) != T):
        raise DpiError(DPI_ERR_INVALID_ARG, "tables / pooling must have one entry per field")
    _check(lib.dpi_lookup_csr(ctypes.c_void_p(plan.handle), _ptr(packed), x_dtype, _ptr(staging), staging_bytes, ptrs,
                              pool, _ptr(offsets), _ptr(ids), _ptr(out), _stream(stream)))


def dpi_plan_destroy(plan: Plan) -> None:
    if plan.handle:
        load().dpi_plan_destroy(ctypes.c_void_p(plan.handle))
        plan.handle = 0
