"""Pins of the oracle's softmax layer (CPU only).

The paper lists softmax among the supported layer types (Sec. 3.1) without a
formula; the oracle takes the normalized exponential across channels.  The
checks below are fixed by closed forms (two classes reduce to the logistic
function, equal inputs to 1/C), invariants (shift invariance, log-ratios equal
input differences, rows sum to one), inputs large enough to overflow a naive
exponential, and torch's CPU softmax in float64 as a library witness for the
channel axis of NCHW tensors.
"""
import math

import numpy as np
import pytest
import torch

import oracle


@pytest.mark.parametrize("a,b", [(0.0, 0.0), (1.0, -2.0), (-3.5, 4.25), (30.0, 0.5), (0.125, 0.0)])
def test_softmax_two_classes_is_logistic(a, b):
    """With two channels, y0 = 1 / (1 + e^(b - a)): the logistic function."""
    y = oracle.softmax_fwd(np.array([[a, b]], dtype=np.float32))
    s0 = 1.0 / (1.0 + math.exp(b - a))
    s1 = 1.0 / (1.0 + math.exp(a - b))
    np.testing.assert_allclose(y[0], [s0, s1], rtol=1e-6, atol=1e-30)


@pytest.mark.parametrize("C,v", [(1, 0.0), (1, -7.0), (7, 3.0), (1000, -2.5), (4096, 1e4)])
def test_softmax_equal_inputs_give_one_over_c(C, v):
    y = oracle.softmax_fwd(np.full((2, C), v, dtype=np.float32))
    assert np.all(y == np.float32(1.0 / C))


def test_softmax_large_inputs_do_not_overflow():
    """exp(1000) overflows double; the max-shifted form gives the exact ratios
    1 : e^-1 : e^-2."""
    y = oracle.softmax_fwd(np.array([[1000.0, 999.0, 998.0]], dtype=np.float32))
    z = 1.0 + math.exp(-1.0) + math.exp(-2.0)
    np.testing.assert_allclose(y[0], [1.0 / z, math.exp(-1.0) / z, math.exp(-2.0) / z], rtol=1e-6)
    y = oracle.softmax_fwd(np.array([[0.0, -1000.0], [-1000.0, 0.0], [1000.0, -1.0]], dtype=np.float32))
    np.testing.assert_array_equal(y, [[1.0, 0.0], [0.0, 1.0], [1.0, 0.0]])


def test_softmax_shift_invariance_and_log_ratios():
    """softmax(x + t) = softmax(x) (inputs chosen so x + t is exact in fp32),
    and log(y_i / y_j) = x_i - x_j."""
    rng = np.random.default_rng(11)
    x = (rng.integers(-64, 64, size=(5, 37)) / 8.0).astype(np.float32)
    y = oracle.softmax_fwd(x)
    np.testing.assert_allclose(oracle.softmax_fwd(x + np.float32(37.5)), y, rtol=2e-7, atol=0)
    lr = np.log(y.astype(np.float64)[:, 1:]) - np.log(y.astype(np.float64)[:, :1])
    np.testing.assert_allclose(lr, (x[:, 1:] - x[:, :1]).astype(np.float64), atol=1e-6)


def test_softmax_rows_sum_to_one_and_keep_order():
    rng = np.random.default_rng(12)
    x = rng.normal(0, 3, size=(8, 100)).astype(np.float32)
    y = oracle.softmax_fwd(x)
    assert np.all(y > 0)
    np.testing.assert_allclose(y.astype(np.float64).sum(axis=1), 1.0, rtol=1e-6)
    assert np.array_equal(np.argsort(x, axis=1, kind="stable"), np.argsort(y, axis=1, kind="stable"))


@pytest.mark.parametrize("shape", [(2, 3, 2, 2), (1, 10, 5, 7), (3, 1, 4, 4), (4, 1000)])
def test_softmax_channel_axis_matches_torch(shape):
    """Across axis 1 of NCHW (each (n, h, w) column separately), as torch's
    softmax(dim=1) in float64."""
    x = np.random.default_rng(13).normal(0, 2, size=shape).astype(np.float32)
    ref = torch.softmax(torch.from_numpy(x).double(), dim=1).numpy()
    np.testing.assert_allclose(oracle.softmax_fwd(x), ref, rtol=1e-6, atol=1e-30)


def test_softmax_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oracle.softmax_fwd(np.zeros((3,), dtype=np.float32))
    assert oracle.softmax_fwd(np.zeros((0, 5), dtype=np.float32)).shape == (0, 5)
