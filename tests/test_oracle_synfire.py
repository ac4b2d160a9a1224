"""Pins of the synfire-term oracle (App. C.1) against hand-computed values,
finite differences and the window's shift structure (CPU only)."""
import math

import numpy as np

import oracle


def test_window_shift_per_layer():
    # layer 0 is the unshifted window; each layer moves both ends by tau_shift
    assert oracle.window(0, 0.3, 1.2, 0.1, 0.2) == (0.1, 1.0)
    for l in range(1, 6):
        a0, b0 = oracle.window(l - 1, 0.3, 1.2, 0.1, 0.2)
        a1, b1 = oracle.window(l, 0.3, 1.2, 0.1, 0.2)
        assert math.isclose(a1 - a0, 0.3) and math.isclose(b1 - b0, 0.3)


def test_temporal_penalty_hand_values():
    # head 0.3, tail 0.7: t = 0.1 is 0.2 early, 0.9 is 0.2 late, 0.5 inside
    t = np.array([0.1, 0.5, 0.9, np.inf])
    val, grad = oracle.temporal_penalty(t, 0.5, 2.0, 0.3, 0.7, 0.25)
    assert math.isclose(val, 0.25 * (0.5 * 0.04 + 2.0 * 0.04), rel_tol=1e-12)
    np.testing.assert_allclose(grad, [0.25 * 2 * 0.5 * -0.2, 0.0, 0.25 * 2 * 2.0 * 0.2, 0.0],
                               rtol=1e-12, atol=1e-15)


def test_temporal_penalty_gradient_finite_difference():
    rng = np.random.default_rng(3)
    t = rng.uniform(-0.5, 1.5, size=(4, 7))
    t[0, 0] = np.inf
    val, grad = oracle.temporal_penalty(t, 0.07, 0.03, 0.25, 0.8, 1.0 / 4)
    h = 1e-6
    for idx in [(0, 1), (1, 3), (2, 5), (3, 6), (1, 0)]:
        tp, tm = t.copy(), t.copy()
        tp[idx] += h
        tm[idx] -= h
        fd = (oracle.temporal_penalty(tp, 0.07, 0.03, 0.25, 0.8, 0.25)[0] -
              oracle.temporal_penalty(tm, 0.07, 0.03, 0.25, 0.8, 0.25)[0]) / (2 * h)
        assert math.isclose(fd, grad[idx], rel_tol=1e-6, abs_tol=1e-9)
    assert grad[0, 0] == 0.0  # silent neuron: no temporal gradient


def test_dead_neuron_hand_values():
    W = np.array([[1.0, 2.0], [3.0, 4.0]])
    t = np.array([[np.inf, 0.5], [np.inf, np.inf]])  # neuron 0 silent twice, neuron 1 once
    val, dW = oracle.dead_neuron_penalty(t, W, 0.1, 0.5)
    assert math.isclose(val, -0.1 * 0.5 * (2 * 3.0 + 1 * 7.0), rel_tol=1e-12)
    np.testing.assert_allclose(dW, -0.05 * np.array([[2, 2], [1, 1]]), rtol=1e-12)


def test_dead_neuron_conv_counts_positions_and_is_linear():
    rng = np.random.default_rng(5)
    W = rng.standard_normal((3, 2, 3, 3))
    t = rng.uniform(0, 1, size=(2, 3, 4, 4))
    t[0, 1, 0, 0] = t[1, 1, 2, 3] = t[1, 2, 1, 1] = np.inf
    val, dW = oracle.dead_neuron_penalty(t, W, 0.2, 1.0 / (2 * 16))
    expect = -0.2 / 32 * (2 * W[1].sum() + W[2].sum())
    assert math.isclose(val, expect, rel_tol=1e-12)
    # Q is linear in W: one finite step recovers each gradient entry
    for idx in [(0, 0, 0, 0), (1, 1, 2, 0), (2, 0, 1, 2)]:
        Wp = W.copy()
        Wp[idx] += 0.5
        assert math.isclose((oracle.dead_neuron_penalty(t, Wp, 0.2, 1 / 32)[0] - val) / 0.5,
                            dW[idx], rel_tol=1e-10, abs_tol=1e-15)
