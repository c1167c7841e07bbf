"""Test-side helpers: build oracle inputs straight from the seeded generator.

Nothing here runs the GPU path.  Rows and ids are regenerated on the CPU from
the counter-based generator, so an oracle input never comes from device
memory written by the library under test.
"""
import numpy as np
import torch

from synth import generate as G
from synth.configs import MEAN


def pooling_codes(cfg):
    return [1 if p == MEAN else 0 for p in G.table_pooling(cfg)]


def sub_problem(cfg, rotation=0, b0=0, b1=None, mapping="literal", lengths=None, ranges=None):
    """Samples [b0, b1) (or the union of ``ranges``) of a workload as a
    self-contained oracle problem.

    Every table is replaced by the rows the sub-batch references (regenerated
    from the generator on the CPU), with ids renumbered into that compact
    table; values and bag structure are unchanged.  The returned "samples"
    lists the original sample index of every row of the sub-problem.
    """
    T, B = cfg.num_tables, cfg.batch
    if ranges is None:
        ranges = [(b0, B if b1 is None else b1)]
    if lengths is None:
        lengths = G.bag_lengths(cfg, rotation)
    offs = G.offsets_from_lengths(lengths)
    sizes = G.table_sizes(cfg)
    samples = np.concatenate([np.arange(lo, hi) for lo, hi in ranges]).astype(np.int64)
    tables, ids, sub_offs, global_ids = [], [], [], []
    for t in range(T):
        n = int(sizes[t])
        cdf = torch.from_numpy(G.zipf_cdf(n, cfg.zipf_s)) if cfg.id_law == "zipf" else None
        parts, lens = [], []
        for lo, hi in ranges:
            s, e = int(offs[t, lo]), int(offs[t, hi])
            parts.append(G.table_ids(cfg, t, n, e - s, rotation, "cpu", mapping, cdf=cdf, start=s))
            lens.append(lengths[t, lo:hi])
        ids_t = torch.cat(parts) if parts else torch.zeros(0, dtype=torch.int64)
        uniq, inv = torch.unique(ids_t, return_inverse=True)
        tables.append(G.table_rows(cfg, t, uniq).numpy())
        ids.append(inv.numpy().astype(np.int32))
        global_ids.append(ids_t.numpy().astype(np.int32))
        L = np.concatenate(lens).astype(np.int64)
        o = np.zeros(len(L) + 1, dtype=np.int64)
        np.cumsum(L, out=o[1:])
        sub_offs.append(o.astype(np.int32))
    return {
        "dims": [cfg.dim(t) for t in range(T)],
        "tables": tables,
        "ids": np.concatenate(ids) if ids else np.zeros(0, np.int32),
        "global_ids": np.concatenate(global_ids) if global_ids else np.zeros(0, np.int32),
        "offsets": np.stack(sub_offs),
        "pooling": pooling_codes(cfg),
        "B": len(samples),
        "samples": samples,
    }


def full_tables(cfg):
    return [G.make_table(cfg, t).numpy() for t in range(cfg.num_tables)]
