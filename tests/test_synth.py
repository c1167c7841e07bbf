"""Seeded generator: determinism, counter-based regeneration and the drawn laws."""
import math

import numpy as np
import pytest
import torch

from synth import configs, generate as G


def test_sizes_in_bounds_and_seeded():
    for cfg in configs.CONFIGS.values():
        s = G.table_sizes(cfg)
        assert len(s) == cfg.num_tables
        assert s.min() >= cfg.rows_lo and s.max() <= cfg.rows_hi
        assert np.array_equal(s, G.table_sizes(cfg))


def test_bag_length_laws():
    L3 = G.bag_lengths(configs.get(3))
    assert L3.min() >= 1 and L3.max() <= 64 and abs(L3.mean() - 10.0) < 0.05
    L4 = G.bag_lengths(configs.get(4))
    assert L4.min() == 0 and L4.max() <= 256 and abs(L4.mean() - 26.98) < 0.1
    assert 300 < (L4 == 0).sum() < 1000          # floor of LogNormal(ln 20, 0.8): P(0) ~ 9e-5
    L5 = G.bag_lengths(configs.get(5))
    assert np.all(L5[:13] == 1)
    frac_empty = (L5[13:] == 0).mean()
    assert abs(frac_empty - 0.05) < 0.005
    assert np.all(G.bag_lengths(configs.get(2)) == 1)
    assert not np.array_equal(G.bag_lengths(configs.get(3), 0), G.bag_lengths(configs.get(3), 1))


def test_values_distribution_and_rounding():
    cfg = configs.get(3)
    assert int(G.table_sizes(cfg)[2]) == 1088
    t = G.make_table(cfg, 2)                 # 1088 x 64 fp16
    x = t.double()
    assert abs(x.mean().item()) < 5e-4
    assert abs(x.std().item() - 0.01) < 0.0002
    c32 = configs.Config(**{**cfg.__dict__, "dtype": configs.F32})
    t32 = G.make_table(c32, 2)
    assert torch.equal(t32.half(), t)


def test_rows_regenerate_exactly():
    cfg = configs.get(2)
    t = 3
    full = G.make_table(cfg, t)
    rows = torch.tensor([0, 5, full.shape[0] - 1, 7, 5], dtype=torch.int64)
    assert torch.equal(G.table_rows(cfg, t, rows), full[rows])


def test_ids_counter_based_and_in_range():
    cfg = configs.get(3)
    n = int(G.table_sizes(cfg)[4])
    a = G.table_ids(cfg, 4, n, 5000, 0)
    b = G.table_ids(cfg, 4, n, 1000, 0, start=2500)
    assert torch.equal(a[2500:3500], b)
    assert a.min() >= 0 and a.max() < n
    batch = G.make_batch(cfg)
    assert batch.ids.dtype == torch.int32 and batch.ids.numel() == batch.total_ids
    base = batch.id_base
    assert torch.equal(batch.ids[base[4]:base[4] + 5000].long(), G.table_ids(cfg, 4, n, 5000, 0))


def test_zipf_rank_frequencies():
    cfg = configs.get(2)
    n = 1000
    ids = G.table_ids(cfg, 0, n, 400_000, 0).numpy()
    counts = np.bincount(ids, minlength=n)
    p = np.arange(1, n + 1, dtype=np.float64) ** -cfg.zipf_s
    p /= p.sum()
    exp = p * len(ids)
    top = slice(0, 50)
    chi2 = (((counts[top] - exp[top]) ** 2) / exp[top]).sum()
    assert chi2 < 100                         # 50 dof; mean 50, sd 10
    assert counts[0] > counts[1] > counts[3]


def test_uniform_ids():
    cfg = configs.get(1)
    ids = G.table_ids(cfg, 0, 1000, 200_000, 0).numpy()
    counts = np.bincount(ids, minlength=1000)
    assert ids.min() >= 0 and ids.max() < 1000
    assert abs(counts.mean() - 200) < 1e-9 and counts.std() < 25


def test_scattered_mapping_is_a_permutation_of_ranks():
    cfg = configs.get(3)
    n = int(G.table_sizes(cfg)[0])
    lit = G.table_ids(cfg, 0, n, 20000, 0, mapping="literal")
    sca = G.table_ids(cfg, 0, n, 20000, 0, mapping="scattered")
    # equal ranks map to equal rows and distinct ranks to distinct rows
    pairs = set(zip(lit.tolist(), sca.tolist()))
    assert len(pairs) == len(set(lit.tolist())) == len(set(sca.tolist()))
