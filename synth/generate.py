"""Seeded synthetic inputs for the fused multi-table lookup.

This module only draws inputs: table sizes, bag lengths, ids and table
values.  It holds none of the lookup's arithmetic (no pooling, no plan), so
both the HIP path and the CPU oracle can consume what it produces.

Every random number is reproducible from ``Config.seed``:
  * sizes, field Poisson means: numpy PCG64 streams keyed by
    ``SeedSequence([seed, purpose])``;
  * bag lengths: a PCG64 stream keyed by ``SeedSequence([seed + 1000*r, 2])``
    for batch rotation ``r``;
  * ids and table values: a counter-based 32-bit integer hash evaluated with
    torch integer ops, so the same element is produced bit-identically on the
    CPU and on the GPU and any single row can be regenerated on demand
    (the oracle does so for the 100-table workload whose tables do not fit in
    host memory).

Value law: four bytes of a hash summed (Irwin-Hall of four discrete
uniforms), centred, scaled to standard deviation 0.01 by one fp32 multiply,
then rounded to fp16 (round-to-nearest-even) for fp16 tables.
Id law: a 53-bit uniform from two hashes, mapped through the inverse CDF of a
bounded Zipf law (fp64 cumulative weights built on the host) or scaled to the
table height for uniform ids.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from functools import lru_cache
from typing import Dict, Iterable, List, Optional, Sequence

import numpy as np
import torch

from .configs import F16, F32, MEAN, SUM, Config

_M32 = 0xFFFFFFFF
_HASH_MUL = 0x45D9F3B          # < 2**27, so x * mul stays below 2**59 in int64
# standard deviation of a sum of four uniform bytes is sqrt(4 * (256**2 - 1) / 12)
VALUE_SCALE = float(np.float32(0.01 / math.sqrt(4.0 * (256 * 256 - 1) / 12.0)))

PURPOSE_SIZES = 0
PURPOSE_VALUES = 1
PURPOSE_LENGTHS = 2
PURPOSE_IDS = 3
PURPOSE_FIELD_MEANS = 4


def _rng(seed: int, purpose: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, purpose])))


def _keys(seed: int, purpose: int, n: int) -> List[int]:
    return [int(k) for k in np.random.SeedSequence([seed, purpose]).generate_state(n, dtype=np.uint32)]


# --------------------------------------------------------------------------------------
# 32-bit counter hash on int64 tensors (values kept in [0, 2**32))
# --------------------------------------------------------------------------------------
def mix32(x: torch.Tensor) -> torch.Tensor:
    """Integer finaliser: xorshift-multiply rounds; input and output in [0, 2**32)."""
    x = x ^ (x >> 16)
    x = (x * _HASH_MUL) & _M32
    x = x ^ (x >> 16)
    x = (x * _HASH_MUL) & _M32
    x = x ^ (x >> 16)
    return x


def counter_hash(ctr: torch.Tensor, k1: int, k2: int) -> torch.Tensor:
    """Keyed hash of a non-negative int64 counter tensor -> [0, 2**32)."""
    lo = ctr & _M32
    hi = ctr >> 32
    a = mix32(lo ^ (k1 & _M32))
    if hi.numel() == 0 or int(hi.max()) == 0:
        b = int(mix32(torch.tensor([k2 & _M32], dtype=torch.int64))[0])
        return mix32((a + b) & _M32)
    b = mix32((hi + (k2 & _M32)) & _M32)
    return mix32((a + b) & _M32)


# --------------------------------------------------------------------------------------
# static per-workload draws
# --------------------------------------------------------------------------------------
def table_sizes(cfg: Config) -> np.ndarray:
    """Row count of every table: clamp(floor(exp(U(ln lo, ln hi))), lo, hi)."""
    if cfg.rows_lo == cfg.rows_hi:
        return np.full(cfg.num_tables, cfg.rows_lo, dtype=np.int64)
    rng = _rng(cfg.seed, PURPOSE_SIZES)
    u = rng.uniform(math.log(cfg.rows_lo), math.log(cfg.rows_hi), cfg.num_tables)
    return np.clip(np.floor(np.exp(u)).astype(np.int64), cfg.rows_lo, cfg.rows_hi)


def table_dims(cfg: Config) -> np.ndarray:
    return np.array([cfg.dim(t) for t in range(cfg.num_tables)], dtype=np.int64)


def table_pooling(cfg: Config) -> List[str]:
    if cfg.pooling == "alternate":
        return [SUM if t % 2 == 0 else MEAN for t in range(cfg.num_tables)]
    return [cfg.pooling] * cfg.num_tables


def field_means(cfg: Config) -> np.ndarray:
    """Per-field Poisson mean for the variable-mean bag law (0 elsewhere)."""
    if cfg.bag.kind != "poisson_var":
        return np.zeros(cfg.num_tables)
    rng = _rng(cfg.seed, PURPOSE_FIELD_MEANS)
    return rng.uniform(cfg.bag.mean_lo, cfg.bag.mean_hi, cfg.num_tables)


def table_bytes(cfg: Config) -> int:
    esize = 2 if cfg.dtype == F16 else 4
    return int((table_sizes(cfg) * table_dims(cfg)).sum()) * esize


# --------------------------------------------------------------------------------------
# bag lengths
# --------------------------------------------------------------------------------------
def bag_lengths(cfg: Config, rotation: int = 0) -> np.ndarray:
    """int64 [T, B]: number of ids in bag (t, b)."""
    T, B = cfg.num_tables, cfg.batch
    rng = _rng(cfg.seed + 1000 * rotation, PURPOSE_LENGTHS)
    lam = field_means(cfg)
    out = np.ones((T, B), dtype=np.int64)
    law = cfg.bag
    for t in range(cfg.onehot_fields, T):
        if law.kind == "poisson":
            x = rng.poisson(law.mean, B)
        elif law.kind == "lognormal":
            x = np.floor(rng.lognormal(math.log(law.mean), law.sigma, B))
        elif law.kind == "poisson_var":
            x = np.maximum(1, rng.poisson(lam[t], B))
            empty = rng.random(B) < law.p_empty
            x = np.where(empty, 0, x)
        else:
            raise ValueError(law.kind)
        out[t] = np.clip(x, law.lo, law.hi).astype(np.int64)
    return out


def offsets_from_lengths(lengths: np.ndarray) -> np.ndarray:
    """int32 [T, B+1] local exclusive prefix of each table's bag lengths."""
    T, B = lengths.shape
    off = np.zeros((T, B + 1), dtype=np.int64)
    np.cumsum(lengths, axis=1, out=off[:, 1:])
    if off[:, -1].max(initial=0) >= 2 ** 31:
        raise ValueError("a table holds 2**31 or more ids")
    return off.astype(np.int32)


# --------------------------------------------------------------------------------------
# ids
# --------------------------------------------------------------------------------------
@lru_cache(maxsize=8)
def _zipf_cdf_cached(n: int, s: float) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return np.cumsum(w)


def zipf_cdf(n: int, s: float) -> np.ndarray:
    """fp64 cumulative weights of a bounded Zipf law over ranks 1..n."""
    return _zipf_cdf_cached(int(n), float(s))


def _uniform53(pos: torch.Tensor, keys: Sequence[int]) -> torch.Tensor:
    h1 = counter_hash(pos, keys[0], keys[1])
    h2 = counter_hash(pos, keys[2], keys[3])
    return ((h1 << 21) | (h2 >> 11)).to(torch.float64) * (2.0 ** -53)


def _scatter_params(n: int, key: int):
    a = (key % n) | 1 if n > 1 else 1
    while math.gcd(a, n) != 1:
        a += 2
    c = (key >> 7) % n if n > 0 else 0
    return a % max(n, 1), c


def table_ids(cfg: Config, t: int, n_rows: int, count: int, rotation: int,
              device: str | torch.device = "cpu", mapping: str = "literal",
              cdf: Optional[torch.Tensor] = None, start: int = 0) -> torch.Tensor:
    """int64 row ids for positions [start, start+count) of table t's id list."""
    keys = _keys(cfg.seed + 1000 * rotation, PURPOSE_IDS, 4 * cfg.num_tables)[4 * t: 4 * t + 4]
    pos = torch.arange(start, start + count, dtype=torch.int64, device=device)
    u = _uniform53(pos, keys)
    if cfg.id_law == "uniform":
        rows = (u * float(n_rows)).to(torch.int64)
        return torch.clamp(rows, max=n_rows - 1)
    if cdf is None:
        cdf = torch.from_numpy(zipf_cdf(n_rows, cfg.zipf_s)).to(device)
    x = u * cdf[-1]
    rank0 = torch.searchsorted(cdf, x, right=True)
    rank0 = torch.clamp(rank0, max=n_rows - 1)
    if mapping == "literal":
        return rank0
    if mapping == "scattered":
        a, c = _scatter_params(n_rows, keys[0] ^ keys[3])
        return (rank0 * a + c) % n_rows
    raise ValueError(mapping)


@dataclass
class Batch:
    cfg: Config
    rotation: int
    lengths: np.ndarray                 # int64 [T, B]
    offsets_host: np.ndarray            # int32 [T, B+1]
    offsets: Optional[torch.Tensor]     # int32 [T, B+1] on device, or None (all one-hot)
    ids: torch.Tensor                   # int32 [total_ids] on device, table-major
    mapping: str = "literal"

    @property
    def nnz(self) -> np.ndarray:
        return self.offsets_host[:, -1].astype(np.int64)

    @property
    def total_ids(self) -> int:
        return int(self.nnz.sum())

    @property
    def id_base(self) -> np.ndarray:
        b = np.zeros(self.cfg.num_tables + 1, dtype=np.int64)
        np.cumsum(self.nnz, out=b[1:])
        return b


def make_batches(cfg: Config, rotations: Iterable[int] = (0,), device: str | torch.device = "cpu",
                 mapping: str = "literal", force_offsets: bool = False) -> List[Batch]:
    """Draw one batch per rotation; ids are generated table by table on ``device``."""
    rotations = list(rotations)
    sizes = table_sizes(cfg)
    lens = {r: bag_lengths(cfg, r) for r in rotations}
    offs = {r: offsets_from_lengths(lens[r]) for r in rotations}
    ids = {r: torch.empty(int(offs[r][:, -1].astype(np.int64).sum()), dtype=torch.int32, device=device)
           for r in rotations}
    for t in range(cfg.num_tables):
        n = int(sizes[t])
        cdf = None
        if cfg.id_law == "zipf":
            cdf = torch.from_numpy(zipf_cdf(n, cfg.zipf_s)).to(device)
        for r in rotations:
            base = int(offs[r][:t, -1].astype(np.int64).sum())
            cnt = int(offs[r][t, -1])
            if cnt:
                ids[r][base: base + cnt] = table_ids(cfg, t, n, cnt, r, device, mapping, cdf).to(torch.int32)
        del cdf
    out = []
    for r in rotations:
        use_off = force_offsets or not cfg.all_onehot
        off_dev = torch.from_numpy(offs[r]).to(device) if use_off else None
        out.append(Batch(cfg, r, lens[r], offs[r], off_dev, ids[r], mapping))
    return out


def make_batch(cfg: Config, rotation: int = 0, device: str | torch.device = "cpu",
               mapping: str = "literal", force_offsets: bool = False) -> Batch:
    return make_batches(cfg, [rotation], device, mapping, force_offsets)[0]


# --------------------------------------------------------------------------------------
# table values
# --------------------------------------------------------------------------------------
def _value_keys(cfg: Config, t: int):
    k = _keys(cfg.seed, PURPOSE_VALUES, 2 * cfg.num_tables)
    return k[2 * t], k[2 * t + 1]


def values_from_counters(cfg: Config, t: int, ctr: torch.Tensor) -> torch.Tensor:
    """Table t's value at element counters ``ctr`` (= row * D + column)."""
    k1, k2 = _value_keys(cfg, t)
    h = counter_hash(ctr, k1, k2)
    s = (h & 255) + ((h >> 8) & 255) + ((h >> 16) & 255) + (h >> 24)
    scale = torch.tensor(VALUE_SCALE, dtype=torch.float32, device=ctr.device)
    v = (s - 510).to(torch.float32) * scale
    return v.to(torch.float16) if cfg.dtype == F16 else v


def table_rows(cfg: Config, t: int, rows: torch.Tensor) -> torch.Tensor:
    """Regenerate the given rows (int64 tensor) of table t: [len(rows), D]."""
    D = cfg.dim(t)
    ctr = rows.to(torch.int64)[:, None] * D + torch.arange(D, dtype=torch.int64, device=rows.device)[None, :]
    return values_from_counters(cfg, t, ctr)


def make_table(cfg: Config, t: int, device: str | torch.device = "cpu",
               n_rows: Optional[int] = None, chunk_elems: int = 1 << 26) -> torch.Tensor:
    n = int(table_sizes(cfg)[t]) if n_rows is None else int(n_rows)
    D = cfg.dim(t)
    dt = torch.float16 if cfg.dtype == F16 else torch.float32
    out = torch.empty((n, D), dtype=dt, device=device)
    flat = out.view(-1)
    total = n * D
    for s in range(0, total, chunk_elems):
        e = min(total, s + chunk_elems)
        ctr = torch.arange(s, e, dtype=torch.int64, device=device)
        flat[s:e] = values_from_counters(cfg, t, ctr)
    return out


def make_tables(cfg: Config, device: str | torch.device = "cpu") -> List[torch.Tensor]:
    return [make_table(cfg, t, device) for t in range(cfg.num_tables)]


def meta(cfg: Config) -> Dict[str, object]:
    """Plain description of the workload's tables (sizes, dims, dtype, pooling)."""
    return {
        "num_rows": table_sizes(cfg),
        "dims": table_dims(cfg),
        "dtype": cfg.dtype,
        "pooling": table_pooling(cfg),
        "out_dtype": cfg.out_dtype,
    }
