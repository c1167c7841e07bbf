"""Pins of the oracle's one-hot input consolidation: a hand-typed example and
the plain transpose of integer-valued matrices (a library routine)."""
import os

import numpy as np

import oracle
from golden_io import GOLDEN


def test_golden_stage():
    rows, ids, T = [], [], None
    with open(os.path.join(GOLDEN, "stage_small.txt")) as f:
        for raw in f:
            tok = raw.split("#", 1)[0].split()
            if not tok:
                continue
            if tok[0] == "fields":
                T = int(tok[1])
            elif tok[0] == "x":
                rows.append([float(v) for v in tok[1:]])
            elif tok[0] == "ids":
                ids.extend(int(v) for v in tok[1:])
    x = np.array(rows, np.float32)
    assert np.array_equal(oracle.stage_onehot(x, T), np.array(ids, np.int32))
    assert np.array_equal(oracle.stage_onehot(x.astype(np.float64), T), np.array(ids, np.int32))


def test_integer_matrix_is_transposed():
    rng = np.random.default_rng(5)
    for dt in (np.int64, np.int32, np.float32):
        x = rng.integers(0, 1 << 20, size=(17, 9)).astype(dt)
        got = oracle.stage_onehot(x, 7)
        assert np.array_equal(got, x[:, :7].T.astype(np.int32).reshape(-1))


def test_out_of_range_integers():
    x = np.array([[-1, 2 ** 31, 2 ** 31 - 1]], np.int64)
    assert list(oracle.stage_onehot(x, 3)) == [-1, -1, 2 ** 31 - 1]


def test_csr_hand_typed():
    # 2 fields, batch 2: field 0 bags {3, 4} {}, field 1 bags {7} {1, 1}
    # packed = offsets of field 0, offsets of field 1, then the ids
    packed = np.array([0, 2, 2, 0, 1, 3, 3, 4, 7, 1, 1], np.int64)
    offs, ids = oracle.stage_csr(packed, 2, 2, 5)
    assert offs.tolist() == [[0, 2, 2], [0, 1, 3]]
    assert ids.tolist() == [3, 4, 7, 1, 1]
    bad = packed.astype(np.float32)
    bad[9] = 1.5
    bad[1] = -2
    offs, ids = oracle.stage_csr(bad, 2, 2, 5)
    assert offs.tolist() == [[0, -1, 2], [0, 1, 3]] and ids.tolist() == [3, 4, 7, -1, 1]
