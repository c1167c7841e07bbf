"""The seeded synthetic workloads of the fused multi-table lookup.

Each workload is a set of sparse fields (one embedding table per field,
§IV-B), a batch size, a bag-length law per field (one-hot or multi-hot,
§IV-B last paragraph: multi-hot fields are described by offsets), an id
distribution over each table's rows and a pooling mode per field.

The shapes stand in for the paper's Criteo (39 fields) and Avazu (24 fields)
inference workloads (§V-A); no record of either dataset is used.  Every
number drawn at random (row counts, bag lengths, ids, table values) comes
from :mod:`synth.generate`, seeded by ``Config.seed``.

Readings of under-specified points:
  * "~N(0, 0.01)" values: standard deviation 0.01.
  * "Zipf(s) over each table's rows": bounded Zipf, P(rank r) ~ r^-s for
    r in [1, n_t]; the literal mapping sends rank r to row r-1 (a
    frequency-sorted vocabulary); the "scattered" variant permutes rows by an
    affine map modulo n_t.
  * log-uniform row counts: n = clamp(floor(exp(U(ln lo, ln hi))), lo, hi).
  * Large workload bag lengths: floor(LogNormal(ln 20, 0.8)) clipped to
    [0, 256] (the floor keeps a few empty bags per batch).
  * Heterogeneous workload: dims [8, 16, 32, 64][t mod 4]; fields 0-12
    one-hot; fields 13-38 multi-hot with a per-field Poisson mean drawn from
    U[1, 40], each bag empty with probability 0.05, otherwise
    max(1, Poisson) clipped at 256.
  * "half tables sum, half mean": even fields sum, odd fields mean.

Workload 6 is the allocation comparison of §V (output-first against
input-first thread allocation at a batch of 65,536 and an embedding dim of
60): 26 one-hot fields of 500,000 rows each, the paper's per-field feature
count of its field sweep.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

F32 = "f32"
F16 = "f16"
SUM = "sum"
MEAN = "mean"


@dataclass(frozen=True)
class BagLaw:
    """How many ids one (sample, field) bag holds."""
    kind: str                      # "onehot" | "poisson" | "lognormal" | "poisson_var"
    mean: float = 0.0              # Poisson mean, or LogNormal median (exp(mu))
    sigma: float = 0.0             # LogNormal sigma
    lo: int = 0                    # clip range
    hi: int = 0
    p_empty: float = 0.0           # probability a bag is forced empty
    mean_lo: float = 0.0           # per-field Poisson mean drawn from U[mean_lo, mean_hi]
    mean_hi: float = 0.0


@dataclass(frozen=True)
class Config:
    key: int
    name: str
    num_tables: int
    batch: int
    rows_lo: int
    rows_hi: int
    dims: Tuple[int, ...]          # cycled over fields: dim_t = dims[t % len(dims)]
    dtype: str                     # table dtype
    out_dtype: str
    id_law: str                    # "uniform" | "zipf"
    zipf_s: float
    pooling: str                   # "sum" | "alternate" (even sum, odd mean)
    onehot_fields: int             # fields [0, onehot_fields) are one-hot
    bag: BagLaw = field(default_factory=lambda: BagLaw("onehot"))
    batches: Tuple[int, ...] = ()  # batch sweep (heterogeneous workload)

    @property
    def seed(self) -> int:
        return 21101000 + self.key

    @property
    def all_onehot(self) -> bool:
        return self.onehot_fields >= self.num_tables

    def dim(self, t: int) -> int:
        return self.dims[t % len(self.dims)]

    def with_batch(self, batch: int) -> "Config":
        return Config(**{**self.__dict__, "batch": batch})

    def with_out(self, out_dtype: str) -> "Config":
        return Config(**{**self.__dict__, "out_dtype": out_dtype})

    def with_dim(self, dim: int) -> "Config":
        return Config(**{**self.__dict__, "dims": (int(dim),)})


TINY = Config(
    key=1, name="tiny-onehot", num_tables=8, batch=256, rows_lo=1000, rows_hi=1000,
    dims=(16,), dtype=F32, out_dtype=F32, id_law="uniform", zipf_s=0.0,
    pooling=SUM, onehot_fields=8)

CTR_ONEHOT = Config(
    key=2, name="ctr-onehot", num_tables=26, batch=4096, rows_lo=10, rows_hi=1_000_000,
    dims=(16,), dtype=F32, out_dtype=F32, id_law="zipf", zipf_s=1.05,
    pooling=SUM, onehot_fields=26)

MULTIHOT = Config(
    key=3, name="multihot", num_tables=26, batch=16384, rows_lo=1_000, rows_hi=5_000_000,
    dims=(64,), dtype=F16, out_dtype=F16, id_law="zipf", zipf_s=1.05,
    pooling=SUM, onehot_fields=0,
    bag=BagLaw("poisson", mean=10.0, lo=1, hi=64))

LARGE = Config(
    key=4, name="large", num_tables=100, batch=65536, rows_lo=100_000, rows_hi=10_000_000,
    dims=(128,), dtype=F16, out_dtype=F16, id_law="zipf", zipf_s=1.1,
    pooling="alternate", onehot_fields=0,
    bag=BagLaw("lognormal", mean=20.0, sigma=0.8, lo=0, hi=256))

HETERO = Config(
    key=5, name="hetero-sweep", num_tables=39, batch=4096, rows_lo=10, rows_hi=10_000_000,
    dims=(8, 16, 32, 64), dtype=F32, out_dtype=F32, id_law="zipf", zipf_s=1.2,
    pooling=SUM, onehot_fields=13,
    bag=BagLaw("poisson_var", lo=0, hi=256, p_empty=0.05, mean_lo=1.0, mean_hi=40.0),
    batches=(1, 16, 128, 512, 4096))

ALLOCATION = Config(
    key=6, name="allocation", num_tables=26, batch=65536, rows_lo=500_000, rows_hi=500_000,
    dims=(60,), dtype=F32, out_dtype=F32, id_law="zipf", zipf_s=1.05,
    pooling=SUM, onehot_fields=26)

CONFIGS = {c.key: c for c in (TINY, CTR_ONEHOT, MULTIHOT, LARGE, HETERO, ALLOCATION)}


def get(key: int, batch: Optional[int] = None, out_dtype: Optional[str] = None,
        dim: Optional[int] = None) -> Config:
    cfg = CONFIGS[int(key)]
    if batch is not None:
        cfg = cfg.with_batch(int(batch))
    if out_dtype is not None:
        cfg = cfg.with_out(out_dtype)
    if dim is not None:
        cfg = cfg.with_dim(int(dim))
    return cfg
