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


def sub_problem(cfg, rotation=0, b0=0, b1=None, mapping="literal", lengths=None):
    """Samples [b0, b1) of a workload as a self-contained oracle problem.

    Every table is replaced by the rows the sub-batch references (regenerated
    from the generator), with ids renumbered into that compact table; values
    and bag structure are unchanged.
    """
    T, B = cfg.num_tables, cfg.batch
    b1 = B if b1 is None else b1
    if lengths is None:
        lengths = G.bag_lengths(cfg, rotation)
    offs = G.offsets_from_lengths(lengths)
    sizes = G.table_sizes(cfg)
    tables, ids, sub_offs, global_ids = [], [], [], []
    for t in range(T):
        s, e = int(offs[t, b0]), int(offs[t, b1])
        ids_t = G.table_ids(cfg, t, int(sizes[t]), e - s, rotation, "cpu", mapping, start=s)
        uniq, inv = torch.unique(ids_t, return_inverse=True)
        tables.append(G.table_rows(cfg, t, uniq).numpy())
        ids.append(inv.numpy().astype(np.int32))
        global_ids.append(ids_t.numpy().astype(np.int32))
        sub_offs.append((offs[t, b0:b1 + 1].astype(np.int64) - s).astype(np.int32))
    return {
        "dims": [cfg.dim(t) for t in range(T)],
        "tables": tables,
        "ids": np.concatenate(ids) if ids else np.zeros(0, np.int32),
        "global_ids": np.concatenate(global_ids) if global_ids else np.zeros(0, np.int32),
        "offsets": np.stack(sub_offs),
        "pooling": pooling_codes(cfg),
        "B": b1 - b0,
    }


def full_tables(cfg):
    return [G.make_table(cfg, t).numpy() for t in range(cfg.num_tables)]
