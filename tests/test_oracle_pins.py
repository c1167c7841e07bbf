"""Pins of the CPU oracle against what the paper and arithmetic fix.

* hand-typed worked examples (tests/golden/, each with its citation);
* the flat index map of the paper's multi-table lookup (§IV-B, Algorithm 1)
  for one-hot fields: a pure copy, so equality is exact;
* a library routine the pooled lookup reduces to: per-field
  torch.nn.functional.embedding_bag in float64, concatenated in field order;
* invariants: empty bag -> 0, one-hot -> the row, mean = sum / L, a repeated
  id counts twice, power-of-two scaling is exact, permuting a bag changes
  nothing, a subset of fields gives the same column block;
* the binary16 decoder on all 65536 bit patterns against numpy's conversion.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from synth import configs, generate as G
from golden_io import load_lookup
from cases import full_tables, pooling_codes, sub_problem


@pytest.mark.parametrize("name", ["lookup_fig5_onehot.txt", "lookup_multihot_mixed.txt"])
def test_golden_lookup(name):
    c = load_lookup(name)
    out = oracle.lookup(c["dims"], c["tables"], c["ids"], c["offsets"], c["pooling"], c["B"],
                        with_mag=False)
    assert np.array_equal(out, c["expected"])


def algorithm1_flat(ids_sample_major, tables, b, k, d):
    """Algorithm 1 (§IV-B) as printed: one loop over all b*k*d output elements."""
    total_elements = b * k * d
    row_width = k * d
    out = np.empty(total_elements, dtype=np.float64)
    flat_tables = [t.astype(np.float64).reshape(-1) for t in tables]
    for idx in range(total_elements):
        row = idx // row_width
        col = idx % row_width
        table_id = col // d
        emb_row = ids_sample_major[row * k + table_id]
        emb_col = col % d
        out[idx] = flat_tables[table_id][emb_row * d + emb_col]
    return out.reshape(b, row_width)


def test_fig5_golden_matches_algorithm1():
    c = load_lookup("lookup_fig5_onehot.txt")
    k, b, d = c["T"], c["B"], c["dims"][0]
    sample_major = c["ids"].reshape(k, b).T.reshape(-1)
    assert np.array_equal(algorithm1_flat(sample_major, c["tables"], b, k, d), c["expected"])


@pytest.mark.parametrize("key,b1", [(1, None), (2, 96)])
def test_onehot_equals_algorithm1(key, b1):
    cfg = configs.get(key)
    if b1 is None:
        tables = full_tables(cfg)
        batch = G.make_batch(cfg)
        ids, B = batch.ids.numpy(), cfg.batch
    else:
        p = sub_problem(cfg, b0=0, b1=b1)
        tables, ids, B = p["tables"], p["ids"], p["B"]
    k, d = cfg.num_tables, cfg.dim(0)
    out = oracle.lookup([d] * k, tables, ids, None, [0] * k, B, with_mag=False)
    sample_major = ids.reshape(k, B).T.reshape(-1)
    assert np.array_equal(out, algorithm1_flat(sample_major, tables, B, k, d))


def embedding_bag_reference(dims, tables, ids, offsets, pooling, B):
    outs, base = [], 0
    for t, d in enumerate(dims):
        off = offsets[t].astype(np.int64)
        n = int(off[-1])
        w = torch.from_numpy(tables[t].astype(np.float64))
        o = F.embedding_bag(torch.from_numpy(ids[base:base + n].astype(np.int64)), w,
                            torch.from_numpy(off), mode="mean" if pooling[t] else "sum",
                            include_last_offset=True)
        outs.append(o.numpy())
        base += n
    return np.concatenate(outs, axis=1)


@pytest.mark.parametrize("key,batch,b1", [(1, None, None), (3, None, 512), (4, None, 48),
                                          (5, 128, None), (5, 512, None), (5, 1, None)])
def test_pooled_equals_embedding_bag(key, batch, b1):
    cfg = configs.get(key, batch=batch)
    p = sub_problem(cfg, b0=0, b1=b1)
    out, mag = oracle.lookup(p["dims"], p["tables"], p["ids"], p["offsets"], p["pooling"], p["B"])
    ref = embedding_bag_reference(p["dims"], p["tables"], p["ids"], p["offsets"], p["pooling"], p["B"])
    # both sums are fp64; only the association order may differ
    assert np.all(np.abs(out - ref) <= 1e-12 * mag + 1e-300)
    if cfg.dtype == configs.F16:
        # fp64 sums of at most 256 binary16 values of this range are exact
        assert np.array_equal(out[:, :] * (np.array(p["pooling"]).repeat(p["dims"]) == 0),
                              ref * (np.array(p["pooling"]).repeat(p["dims"]) == 0))


def _random_case(rng, T=3, B=5, dtype=np.float32, max_len=6, pooling=None):
    dims = [int(rng.choice([1, 2, 3, 4, 8])) * (2 if dtype == np.float16 else 1) for _ in range(T)]
    rows = [int(rng.integers(1, 9)) for _ in range(T)]
    tables = [(rng.integers(-64, 64, size=(rows[t], dims[t])) / 16.0).astype(dtype) for t in range(T)]
    lens = rng.integers(0, max_len + 1, size=(T, B))
    offs = np.zeros((T, B + 1), dtype=np.int32)
    offs[:, 1:] = np.cumsum(lens, axis=1)
    ids = np.concatenate([rng.integers(0, rows[t], size=int(offs[t, -1])) for t in range(T)]).astype(np.int32)
    pooling = pooling if pooling is not None else [int(x) for x in rng.integers(0, 2, T)]
    return dims, tables, ids, offs, pooling, B


def test_empty_bags_are_zero():
    rng = np.random.default_rng(1)
    dims, tables, ids, offs, pool, B = _random_case(rng)
    offs[:, :] = 0
    for pooling in ([0] * 3, [1] * 3):
        out = oracle.lookup(dims, tables, np.zeros(0, np.int32), offs, pooling, B, with_mag=False)
        assert np.array_equal(out, np.zeros_like(out))


def test_one_hot_bag_is_the_row():
    rng = np.random.default_rng(2)
    for dtype in (np.float32, np.float16):
        dims, tables, _, _, _, B = _random_case(rng, dtype=dtype)
        ids = np.concatenate([rng.integers(0, tables[t].shape[0], size=B) for t in range(3)]).astype(np.int32)
        offs = np.tile(np.arange(B + 1, dtype=np.int32), (3, 1))
        for pooling in ([0] * 3, [1] * 3):
            out = oracle.lookup(dims, tables, ids, offs, pooling, B, with_mag=False)
            col = 0
            for t, d in enumerate(dims):
                rows = tables[t][ids[t * B:(t + 1) * B]].astype(np.float64)
                assert np.array_equal(out[:, col:col + d], rows)
                col += d


def test_mean_is_sum_over_length():
    rng = np.random.default_rng(3)
    dims, tables, ids, offs, _, B = _random_case(rng, max_len=9)
    s = oracle.lookup(dims, tables, ids, offs, [0] * 3, B, with_mag=False)
    m = oracle.lookup(dims, tables, ids, offs, [1] * 3, B, with_mag=False)
    lens = np.diff(offs.astype(np.int64), axis=1)          # [T, B]
    col = 0
    for t, d in enumerate(dims):
        L = lens[t][:, None].astype(np.float64)
        expect = np.where(L > 0, s[:, col:col + d] / np.maximum(L, 1), 0.0)
        assert np.array_equal(m[:, col:col + d], expect)
        col += d


def test_repeated_id_counts_twice_and_scaling_is_exact():
    rng = np.random.default_rng(4)
    dims, tables, _, _, _, B = _random_case(rng, T=2)
    ids = np.concatenate([np.repeat(rng.integers(0, tables[t].shape[0], size=B), 2) for t in range(2)]).astype(np.int32)
    offs = np.tile(np.arange(0, 2 * B + 1, 2, dtype=np.int32), (2, 1))
    out = oracle.lookup(dims, tables, ids, offs, [0, 0], B, with_mag=False)
    col = 0
    for t, d in enumerate(dims):
        rows = tables[t][ids[t * 2 * B:(t + 1) * 2 * B:2]].astype(np.float64)
        assert np.array_equal(out[:, col:col + d], 2.0 * rows)
        col += d
    scaled = [(t.astype(np.float64) * 8.0).astype(t.dtype) for t in tables]
    out8 = oracle.lookup(dims, scaled, ids, offs, [0, 0], B, with_mag=False)
    assert np.array_equal(out8, 8.0 * out)


def test_permuting_a_bag_changes_nothing():
    rng = np.random.default_rng(5)
    dims, tables, ids, offs, pool, B = _random_case(rng, dtype=np.float16, max_len=12)
    perm = ids.copy()
    base = 0
    for t in range(3):
        for b in range(B):
            s, e = base + offs[t, b], base + offs[t, b + 1]
            perm[s:e] = rng.permutation(perm[s:e])
        base += offs[t, -1]
    a = oracle.lookup(dims, tables, ids, offs, pool, B, with_mag=False)
    b = oracle.lookup(dims, tables, perm, offs, pool, B, with_mag=False)
    assert np.array_equal(a, b)   # binary16 sums are exact in fp64


def test_subset_of_fields_gives_same_columns():
    rng = np.random.default_rng(6)
    dims, tables, ids, offs, pool, B = _random_case(rng, T=4)
    full = oracle.lookup(dims, tables, ids, offs, pool, B, with_mag=False)
    nnz = offs[:, -1].astype(np.int64)
    base = np.concatenate([[0], np.cumsum(nnz)])
    col = np.concatenate([[0], np.cumsum(dims)])
    for t in range(4):
        one = oracle.lookup([dims[t]], [tables[t]], ids[base[t]:base[t + 1]], offs[t:t + 1], [pool[t]], B,
                            with_mag=False)
        assert np.array_equal(one, full[:, col[t]:col[t + 1]])


def test_magnitude_is_sum_of_abs():
    rng = np.random.default_rng(7)
    dims, tables, ids, offs, pool, B = _random_case(rng)
    _, mag = oracle.lookup(dims, tables, ids, offs, pool, B)
    abs_tables = [np.abs(t) for t in tables]
    out_abs = oracle.lookup(dims, abs_tables, ids, offs, pool, B, with_mag=False)
    assert np.array_equal(mag, out_abs)


def test_binary16_decode_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    table = bits.view(np.float16).reshape(-1, 2)          # 32768 rows of dim 2
    n = table.shape[0]
    ids = np.arange(n, dtype=np.int32)
    out = oracle.lookup([2], [table], ids, None, [0], n, with_mag=False)
    ref = table.astype(np.float64)
    # value equality fixes the sign of every non-zero pattern; a sum that
    # starts from +0 legitimately turns -0 into +0
    assert np.array_equal(out, ref, equal_nan=True)


def test_out_of_range_id_is_reported():
    t = np.zeros((3, 2), dtype=np.float32)
    with pytest.raises(oracle.OracleError) as e:
        oracle.lookup([2], [t], np.array([3], np.int32), None, [0], 1)
    assert e.value.code == oracle.BAD_ID
