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


def test_dcn_magnitude_hand_typed():
    """The magnitudes are the two networks run on absolute values (inputs, weights,
    biases) without the ReLU: the scale of the fp32 error bounds of the GPU head.
    Worked by hand for one cross layer and a two-layer MLP, d = 2."""
    x0 = np.array([[1.0, -2.0]])
    W = np.array([[0.5, 0.5], [1.0, -1.0]])
    b = np.array([0.25, 2.0])
    # signed:   x0 W^T = [0.5 - 1, 1 + 2] = [-0.5, 3]; + b = [-0.25, 5]
    #           x1 = x0 * [-0.25, 5] + x0 = [0.75, -12]
    # absolute: |x0| |W|^T = [0.5 + 1, 1 + 2] = [1.5, 3]; + |b| = [1.75, 5]
    #           |x0| * [1.75, 5] + |x0| = [2.75, 12]
    V1 = np.array([[1.0, 1.0], [-1.0, 0.0], [0.0, 0.5]])
    c1 = np.array([0.0, 0.0, -2.0])
    V2 = np.array([[1.0, -1.0, 0.5]])
    c2 = np.array([-1.0])
    # signed:   relu([1 - 2, -1, -1] + [0, 0, -2]) = [0, 0, 0]; relu(0 - 1) = [0]
    # absolute: [1 + 2, 1, 1] + [0, 0, 2] = [3, 1, 3]; 3 + 1 + 1.5 + 1 = [6.5]
    x, h, ax, ah = oracle.dcn_forward(x0, [W], [b], [V1, V2], [c1, c2])
    assert np.array_equal(x, np.array([[0.75, -12.0]]))
    assert np.array_equal(ax, np.array([[2.75, 12.0]]))
    assert np.array_equal(h, np.array([[0.0]]))
    assert np.array_equal(ah, np.array([[6.5]]))


def _random_head(rng, B=4, d=5, L=2, mlp=(7, 3)):
    cw = [rng.standard_normal((d, d)) for _ in range(L)]
    cb = [rng.standard_normal(d) for _ in range(L)]
    mw, mb, prev = [], [], d
    for h in mlp:
        mw.append(rng.standard_normal((h, prev)))
        mb.append(rng.standard_normal(h))
        prev = h
    return rng.standard_normal((B, d)), cw, cb, mw, mb


def test_dcn_magnitude_identity_on_nonnegative_inputs():
    """With non-negative inputs, weights and biases nothing cancels and no ReLU
    cuts, so each magnitude is the network's own output, bit for bit."""
    rng = np.random.default_rng(4)
    x0, cw, cb, mw, mb = _random_head(rng)
    x0, cw, cb, mw, mb = np.abs(x0), [np.abs(w) for w in cw], [np.abs(v) for v in cb], \
        [np.abs(w) for w in mw], [np.abs(v) for v in mb]
    x, h, ax, ah = oracle.dcn_forward(x0, cw, cb, mw, mb)
    assert np.array_equal(ax, x)
    assert np.array_equal(ah, h)


def test_dcn_magnitude_sign_invariance_and_bound():
    """Flipping the signs of any inputs, weights and biases leaves the magnitudes
    unchanged, and each magnitude bounds its output (triangle inequality)."""
    rng = np.random.default_rng(6)
    x0, cw, cb, mw, mb = _random_head(rng)
    x, h, ax, ah = oracle.dcn_forward(x0, cw, cb, mw, mb)
    assert np.all(ax >= np.abs(x)) and np.all(ah >= np.abs(h))

    def flip(a):
        return a * np.where(rng.random(a.shape) < 0.5, -1.0, 1.0)

    _, _, ax2, ah2 = oracle.dcn_forward(flip(x0), [flip(w) for w in cw], [flip(v) for v in cb],
                                        [flip(w) for w in mw], [flip(v) for v in mb])
    assert np.array_equal(ax2, ax)
    assert np.array_equal(ah2, ah)
