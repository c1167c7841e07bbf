"""Pins of the oracle's second-order FM term (§IV-D, DeepFM's explicit
interaction): a hand-typed example, the pairwise dot-product form on random
inputs, and closed forms."""
import os

import numpy as np
import pytest

import oracle
from golden_io import GOLDEN


def load_fm(name, with_mag=False):
    rows, expect, mags, T, D = [], [], [], None, None
    with open(os.path.join(GOLDEN, name)) as f:
        for raw in f:
            line = raw.split("#", 1)[0].split()
            if not line:
                continue
            if line[0] == "fields":
                T = int(line[1])
            elif line[0] == "dim":
                D = int(line[1])
            elif line[0] == "row":
                rows.append([float(x) for x in line[1:]])
            elif line[0] == "expect":
                expect.append(float(line[1]))
            elif line[0] == "mag":
                mags.append(float(line[1]))
    if with_mag:
        return np.array(rows, np.float32), np.array(expect), np.array(mags), T, D
    return np.array(rows, np.float32), np.array(expect), T, D


def pairwise(e, T, D):
    """The term's defining form: sum over field pairs t < u of <e_t, e_u>."""
    B = e.shape[0]
    v = e[:, : T * D].astype(np.float64).reshape(B, T, D)
    out = np.zeros(B)
    for t in range(T):
        for u in range(t + 1, T):
            out += np.einsum("bc,bc->b", v[:, t], v[:, u])
    return out


def pairwise_magnitude(e, T, D):
    """The magnitude's defining form: per column, the sum of the squares plus the
    sum over field pairs t < u of |e_tc| |e_uc| (the scale of the fp32 error of
    squaring the column sum and subtracting the sum of squares)."""
    B = e.shape[0]
    v = e[:, : T * D].astype(np.float64).reshape(B, T, D)
    out = np.zeros(B)
    for b in range(B):
        for c in range(D):
            col = v[b, :, c]
            out[b] += sum(x * x for x in col)
            for t in range(T):
                for u in range(t + 1, T):
                    out[b] += abs(col[t]) * abs(col[u])
    return out


def test_golden_fm():
    e, expect, T, D = load_fm("fm_small.txt")
    out = oracle.fm_second_order(e, T, D, with_mag=False)
    assert np.array_equal(out, expect)


def test_golden_fm_magnitude():
    e, expect, mags, T, D = load_fm("fm_small.txt", with_mag=True)
    out, mag = oracle.fm_second_order(e, T, D)
    assert np.array_equal(out, expect)
    assert np.array_equal(mag, mags)


@pytest.mark.parametrize("T,D,dtype", [(2, 1, np.float32), (3, 5, np.float32), (7, 16, np.float16),
                                       (26, 8, np.float32)])
def test_magnitude_equals_pairwise_form(T, D, dtype):
    rng = np.random.default_rng(T * 7 + D)
    e = (rng.standard_normal((5, T * D + 2)) * 0.1).astype(dtype)
    _, mag = oracle.fm_second_order(e, T, D)
    assert np.allclose(mag, pairwise_magnitude(e, T, D), rtol=1e-12, atol=0)


def test_magnitude_closed_forms():
    rng = np.random.default_rng(8)
    # non-negative values: the magnitude exceeds the term by exactly the sum of squares
    e = (rng.integers(0, 16, size=(4, 15)) / 8).astype(np.float32)
    out, mag = oracle.fm_second_order(e, 5, 3)
    sq = (e.astype(np.float64) ** 2).sum(axis=1)
    assert np.array_equal(mag - out, sq)
    # signs do not change the magnitude
    flip = np.where(rng.random(e.shape) < 0.5, -1, 1).astype(np.float32)
    _, mag2 = oracle.fm_second_order(e * flip, 5, 3)
    assert np.array_equal(mag2, mag)
    # one field: the magnitude is the squared norm of the row
    _, m1 = oracle.fm_second_order(e[:, :3], 1, 3)
    assert np.array_equal(m1, (e[:, :3].astype(np.float64) ** 2).sum(axis=1))


@pytest.mark.parametrize("T,D,dtype", [(2, 1, np.float32), (3, 5, np.float32), (7, 16, np.float16),
                                       (26, 8, np.float32)])
def test_equals_pairwise_dot_products(T, D, dtype):
    rng = np.random.default_rng(T * 100 + D)
    e = (rng.standard_normal((9, T * D + 3)) * 0.1).astype(dtype)   # 3 extra columns are ignored
    out, mag = oracle.fm_second_order(e, T, D)
    ref = pairwise(e, T, D)
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-15)
    assert np.all(mag >= np.abs(out) - 1e-15)


def test_closed_forms():
    rng = np.random.default_rng(3)
    v = rng.integers(-8, 8, size=6).astype(np.float32) / 4
    # one field: no pair
    assert np.all(oracle.fm_second_order(v[None, :], 1, 6, with_mag=False) == 0)
    # T equal fields: T(T-1)/2 |v|^2
    for T in (2, 3, 5):
        e = np.tile(v, T)[None, :]
        assert oracle.fm_second_order(e, T, 6, with_mag=False)[0] == T * (T - 1) / 2 * float(v @ v)
    # orthogonal fields: zero
    e = np.array([[1, 0, 0, 0, 2, 0, 0, 0, -3]], np.float32)
    assert oracle.fm_second_order(e, 3, 3, with_mag=False)[0] == 0.0
    # scaling every value by 2^k scales the term by 4^k exactly
    e = (rng.integers(-16, 16, size=(4, 12)) / 8).astype(np.float32)
    a = oracle.fm_second_order(e, 4, 3, with_mag=False)
    b = oracle.fm_second_order(e * 4, 4, 3, with_mag=False)
    assert np.array_equal(b, a * 16)


def test_rejects_bad_arguments():
    e = np.zeros((2, 4), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.fm_second_order(e, 3, 2)          # 3 * 2 > 4 columns
    with pytest.raises(oracle.OracleError):
        oracle.fm_second_order(e, 0, 2)
