"""torch-facing convenience over the C ABI: device memory and streams only.

FusedLookup keeps a set of field tables and, per batch, runs dpi_plan then
dpi_lookup on the current (or given) stream into a [B, sum dim] tensor.
"""
from __future__ import annotations

from typing import Optional, Sequence

import torch

from . import dpi

_DT = {torch.float32: dpi.DPI_F32, torch.float16: dpi.DPI_F16}
_TORCH = {dpi.DPI_F32: torch.float32, dpi.DPI_F16: torch.float16}


class FusedLookup:
    """The tables of a set of fields and one workspace, reused by every plan():
    each plan supersedes the one before it (a lookup or export with an earlier
    plan raises).  To keep several plans in flight, give each its own
    workspace through dpi.dpi_plan."""

    def __init__(self, tables: Sequence[torch.Tensor], pooling: Optional[Sequence[int]] = None,
                 out_dtype: torch.dtype = torch.float32, num_rows: Optional[Sequence[int]] = None,
                 chunk_rows: int = 0, item_cost_k: int = 0, flags: int = 0):
        self.tables = list(tables)
        self.T = len(self.tables)
        self.dims = [int(t.shape[1]) for t in self.tables]
        self.dtypes = [_DT[t.dtype] for t in self.tables]
        rows = num_rows if num_rows is not None else [int(t.shape[0]) for t in self.tables]
        self.meta = dpi.make_meta(rows, self.dims, self.dtypes)
        self.pooling = list(pooling) if pooling is not None else None
        self.out_dtype = out_dtype
        self.chunk_rows, self.item_cost_k, self.flags = chunk_rows, item_cost_k, flags
        self.device = self.tables[0].device
        self._ws = None
        # host arrays handed to every lookup (built once)
        self._table_ptrs = dpi.table_array(self.tables)
        self._pool = None if self.pooling is None else dpi.pooling_array(self.pooling)

    @property
    def total_dim(self) -> int:
        return sum(self.dims)

    def opts(self, num_waves: int = 0) -> dpi.dpi_plan_opts:
        return dpi.make_opts(self.chunk_rows, self.item_cost_k, num_waves, _DT[self.out_dtype], self.flags)

    def workspace(self, batch: int, total_ids: int, opts) -> torch.Tensor:
        need = dpi.dpi_plan_workspace_bytes(self.T, batch, total_ids, max(self.dims), opts)
        if need == 0:
            raise dpi.DpiError(dpi.DPI_ERR_INVALID_ARG, "workspace size query failed")
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        return self._ws

    def plan(self, offsets: Optional[torch.Tensor], batch: int, total_ids: int, num_waves: int = 0,
             stream=None) -> dpi.Plan:
        o = self.opts(num_waves)
        ws = self.workspace(batch, total_ids, o)
        return dpi.dpi_plan(self.meta, offsets, batch, total_ids, o, ws, stream=stream)

    def lookup(self, plan: dpi.Plan, ids: torch.Tensor, offsets: Optional[torch.Tensor],
               out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        if out is None:
            out = torch.empty((plan.batch, self.total_dim), dtype=self.out_dtype, device=self.device)
        dpi.dpi_lookup(plan, self._table_ptrs, ids, offsets, self._pool, out, stream=stream)
        return out

    def __call__(self, ids: torch.Tensor, offsets: Optional[torch.Tensor], batch: int,
                 out: Optional[torch.Tensor] = None, num_waves: int = 0, stream=None) -> torch.Tensor:
        p = self.plan(offsets, batch, int(ids.numel()), num_waves, stream)
        return self.lookup(p, ids, offsets, out, stream)
