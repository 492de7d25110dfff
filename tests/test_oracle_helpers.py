"""Pins of the oracle's small helpers against values fixed by their definitions.

rms_norm (the decode block's RMSNorm, Sec. 3.8), rms_normalise (the gain-free
norm of Eq. 13), the logistic gate of Eq. 12, the affine map y = x W^T + b used
by every projection, and the error metric the parity tests use.
"""
import math

import numpy as np
import pytest

import oracle
from oracle.layer import AFFINE_EPS, linear, rms_normalise, sigmoid


def test_rms_norm_hand_example_and_gain():
    # x = (3, 4): mean square 12.5, so x / sqrt(12.5) = (0.84853, 1.13137)
    got = oracle.rms_norm(np.array([[3.0, 4.0]]), np.array([1.0, 1.0]), 0.0)
    np.testing.assert_allclose(got, [[3 / math.sqrt(12.5), 4 / math.sqrt(12.5)]], rtol=1e-15)
    # the gain multiplies channel by channel; eps enters under the root
    got = oracle.rms_norm(np.array([[3.0, 4.0]]), np.array([2.0, -1.0]), 0.5)
    np.testing.assert_allclose(got, [[6 / math.sqrt(13.0), -4 / math.sqrt(13.0)]], rtol=1e-15)


def test_rms_norm_unit_rms_and_scale_invariance():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 96)) * 7.0
    y = oracle.rms_norm(x, np.ones(96), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-13)
    np.testing.assert_allclose(oracle.rms_norm(3.5 * x, np.ones(96), 0.0), y, rtol=1e-13)
    # rows are normalised independently
    np.testing.assert_allclose(oracle.rms_norm(x[2:3], np.ones(96), 0.0), y[2:3], rtol=1e-15)


def test_rms_normalise_has_no_gain_and_its_own_eps():
    x = np.array([[3.0, 4.0], [0.0, 0.0]])
    got = rms_normalise(x)
    np.testing.assert_allclose(got[0], [3 / math.sqrt(12.5 + AFFINE_EPS), 4 / math.sqrt(12.5 + AFFINE_EPS)],
                               rtol=1e-15)
    np.testing.assert_array_equal(got[1], [0.0, 0.0])  # eps keeps an all-zero token finite
    assert AFFINE_EPS == 1e-6


def test_sigmoid_special_values_and_symmetry():
    np.testing.assert_allclose(sigmoid(np.array([0.0, math.log(3.0), -math.log(3.0)])), [0.5, 0.75, 0.25],
                               rtol=1e-15)
    z = np.linspace(-30, 30, 121)
    np.testing.assert_allclose(sigmoid(z) + sigmoid(-z), 1.0, rtol=1e-15)
    # no overflow at the extremes, and the limits are reached
    big = sigmoid(np.array([-800.0, 800.0]))
    assert np.all(np.isfinite(big)) and big[0] == 0.0 and big[1] == 1.0
    # derivative identity sigma' = sigma (1 - sigma), by central differences
    h = 1e-5
    zz = np.array([-2.0, 0.3, 4.0])
    fd = (sigmoid(zz + h) - sigmoid(zz - h)) / (2 * h)
    np.testing.assert_allclose(fd, sigmoid(zz) * (1 - sigmoid(zz)), rtol=1e-8)


def test_linear_against_explicit_sums():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 4))
    w = rng.standard_normal((5, 4))  # [out, in]
    b = rng.standard_normal(5)
    want = np.array([[sum(x[r, i] * w[o, i] for i in range(4)) + b[o] for o in range(5)] for r in range(3)])
    np.testing.assert_allclose(linear(x, w, b), want, rtol=1e-13)
    np.testing.assert_allclose(linear(x, w, None), want - b, rtol=1e-13, atol=1e-15)


def test_max_rel_err_is_the_infinity_norm_ratio():
    assert oracle.max_rel_err([1.0, -2.0], [1.0, -2.0]) == 0.0
    assert oracle.max_rel_err([1.0, -2.2], [1.0, -2.0]) == pytest.approx(0.1)
    assert oracle.max_rel_err([0.5, 4.0], [1.0, -4.0]) == pytest.approx(2.0)
    assert oracle.max_rel_err([0.25], [0.0]) == 0.25  # zero reference: absolute error
    assert oracle.max_rel_err(np.zeros((0, 3)), np.zeros((0, 3))) == 0.0
    with pytest.raises(ValueError):
        oracle.max_rel_err([1.0], [1.0, 2.0])
