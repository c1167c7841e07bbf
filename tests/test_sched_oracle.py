"""Pins of the oracle's breadth-first launch queue (Algorithm 2, §IV-E) and of
its interaction-module forward (cross network and MLP) by invariants, a
hand-typed queue and closed forms."""
import numpy as np
import pytest

import oracle


def test_hand_typed_queues():
    # more implicit operators: implicit first, then alternating, implicit tail
    assert oracle.breadth_first_order(2, 4) == [("I", 0), ("E", 0), ("I", 1), ("E", 1), ("I", 2), ("I", 3)]
    # more explicit operators, and a tie: explicit first
    assert oracle.breadth_first_order(3, 1) == [("E", 0), ("I", 0), ("E", 1), ("E", 2)]
    assert oracle.breadth_first_order(2, 2) == [("E", 0), ("I", 0), ("E", 1), ("I", 1)]
    assert oracle.breadth_first_order(0, 2) == [("I", 0), ("I", 1)]
    assert oracle.breadth_first_order(0, 0) == []


@pytest.mark.parametrize("ne,ni", [(n, m) for n in range(7) for m in range(7)])
def test_queue_invariants(ne, ni):
    q = oracle.breadth_first_order(ne, ni)
    # every operator exactly once, each module in its own order
    assert [i for k, i in q if k == "E"] == list(range(ne))
    assert [j for k, j in q if k == "I"] == list(range(ni))
    # while both modules have operators left, consecutive entries alternate modules
    m = min(ne, ni)
    kinds = [k for k, _ in q]
    assert all(kinds[i] != kinds[i + 1] for i in range(2 * m - 1))
    # the tail holds only the longer module
    assert len(set(kinds[2 * m:])) <= 1


def test_dcn_closed_forms():
    rng = np.random.default_rng(1)
    B, d = 5, 6
    x0 = rng.standard_normal((B, d))
    # W = 0, b = 1: every cross layer adds x0, so L layers give (L + 1) x0
    L = 3
    x, _, _, _ = oracle.dcn_forward(x0, [np.zeros((d, d))] * L, [np.ones(d)] * L, [], [])
    assert np.allclose(x, (L + 1) * x0, rtol=0, atol=1e-12)
    # W = 0, b = 0: the cross layers keep x0
    x, _, _, _ = oracle.dcn_forward(x0, [np.zeros((d, d))] * 2, [np.zeros(d)] * 2, [], [])
    assert np.array_equal(x, x0)
    # identity MLP layer with zero bias is the ReLU; a negative bias shifts it
    _, h, _, _ = oracle.dcn_forward(x0, [], [], [np.eye(d)], [np.zeros(d)])
    assert np.array_equal(h, np.maximum(0, x0))
    _, h, _, _ = oracle.dcn_forward(x0, [], [], [np.eye(d)], [-np.ones(d)])
    assert np.array_equal(h, np.maximum(0, x0 - 1))


def test_dcn_hand_typed():
    # one cross layer, d = 2: x1 = x0 * (x0 W^T + b) + x0
    x0 = np.array([[1.0, 2.0]])
    W = np.array([[0.5, 0.0], [1.0, -1.0]])      # x0 W^T = [0.5, -1]
    b = np.array([0.25, 2.0])                      # + b  = [0.75, 1]
    x, _, _, _ = oracle.dcn_forward(x0, [W], [b], [], [])
    assert np.array_equal(x, np.array([[1.75, 4.0]]))  # [1*0.75 + 1, 2*1 + 2]
    # one MLP layer to 3 units: relu([1*1 + 2*1, 1*(-1) + 0, 2*0.5] + [0, 0, -2])
    V = np.array([[1.0, 1.0], [-1.0, 0.0], [0.0, 0.5]])
    c = np.array([0.0, 0.0, -2.0])
    _, h, _, _ = oracle.dcn_forward(x0, [], [], [V], [c])
    assert np.array_equal(h, np.array([[3.0, 0.0, 0.0]]))
