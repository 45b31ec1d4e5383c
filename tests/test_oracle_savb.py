"""Pins of the oracle's SAVB gate (Sec. 3.2, Eqs. 2 and 3), CPU only.

  * the feature on a hand-worked example: the mean of the preceding text
    states, then the final one; a single text token gives a zero mean;
  * the MLP on a hand-worked example with one negative pre-activation (the
    ReLU zeroes it) and biases on both layers;
  * two classes: p_exit is the logistic of z_1 - z_0, and the decision at
    p_exit == theta exactly is an exit (">=").
"""

import numpy as np
import pytest

import oracle


def test_feature_hand_worked():
    rows = np.array([[1.0, 2.0], [3.0, 4.0], [5.0, 6.0]])
    np.testing.assert_array_equal(oracle.savb_gate_feature(rows), [2.0, 3.0, 5.0, 6.0])
    np.testing.assert_array_equal(oracle.savb_gate_feature(rows[2:]), [0.0, 0.0, 5.0, 6.0])
    with pytest.raises(ValueError):
        oracle.savb_gate_feature(np.zeros((0, 2)))


def test_mlp_hand_worked():
    # d = 1: x = [mean of 2 and 4; 10] = [3, 10]
    rows = np.array([[2.0], [4.0], [10.0]])
    w1 = np.array([[1.0, 0.0], [0.0, -1.0], [1.0, 1.0]])   # pre-activations 3, -10, 13
    b1 = np.array([0.5, 0.0, -1.0])                       # -> 3.5, -10 (relu 0), 12
    w2 = np.array([[1.0, 0.0, 0.0], [0.0, 0.0, 1.0]])      # z = [3.5 + b, 12 + b]
    b2 = np.array([0.25, -0.25])
    p, ex, x, z = oracle.savb_gate(rows, w1, b1, w2, b2, 0.5)
    np.testing.assert_array_equal(x, [3.0, 10.0])
    np.testing.assert_array_equal(z, [3.75, 11.75])
    assert p == pytest.approx(1.0 / (1.0 + np.exp(-8.0)), rel=1e-15)
    assert ex


def test_two_class_logistic_and_threshold_tie():
    rng = np.random.default_rng(0)
    rows = rng.normal(size=(5, 4))
    w1, b1 = rng.normal(size=(6, 8)), rng.normal(size=6)
    w2, b2 = rng.normal(size=(2, 6)), rng.normal(size=2)
    p, ex, x, z = oracle.savb_gate(rows, w1, b1, w2, b2, 0.3)
    assert p == pytest.approx(1.0 / (1.0 + np.exp(z[0] - z[1])), rel=1e-14)
    assert ex == (p >= 0.3)
    # equal class logits: p_exit = 1/2 exactly, and theta = 1/2 exits
    p2, ex2, _, _ = oracle.savb_gate(rows, w1, b1, np.zeros((2, 6)), np.zeros(2), 0.5)
    assert p2 == 0.5 and ex2
    _, ex3, _, _ = oracle.savb_gate(rows, w1, b1, np.zeros((2, 6)), np.zeros(2), np.nextafter(0.5, 1))
    assert not ex3
