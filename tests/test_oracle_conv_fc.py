"""Pins of the oracle's convolution and fully-connected layers (CPU only).

Each check is fixed by something other than the oracle itself: a hand-derived
fixture, a closed form, an invariant of the definition, or a library routine
(torch's CPU conv2d / numpy matmul in float64) that the definition reduces to.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from golden_io import load


def _rand(shape, seed, lo=-1.0, hi=1.0):
    return np.random.default_rng(seed).uniform(lo, hi, shape).astype(np.float32)


# ---------------------------------------------------------------- fixtures
def test_conv_golden_stride1_bias():
    g = load("conv_3x3_k2x2.txt")
    y = oracle.conv2d_fwd(g["x"], g["w"], g["bias_a"])
    np.testing.assert_array_equal(y, g["y_a"].astype(np.float32))


def test_conv_golden_stride2_pad1():
    g = load("conv_3x3_k2x2.txt")
    y = oracle.conv2d_fwd(g["x"], g["w"], None, stride=(2, 2), pad=(1, 1))
    np.testing.assert_array_equal(y, g["y_b"].astype(np.float32))


# ---------------------------------------------------------------- shapes
@pytest.mark.parametrize("H,R,s,p,expect", [
    (227, 11, 4, 0, 55),    # AlexNet conv1
    (27, 5, 1, 2, 27),      # AlexNet conv2
    (13, 3, 1, 1, 13),      # AlexNet conv3-5
    (28, 5, 1, 0, 24),      # LeNet conv1
    (12, 5, 1, 0, 8),       # LeNet conv2
    (32, 5, 1, 2, 32),      # CIFAR convs
    (224, 7, 2, 3, 112),    # stem: (224+6-7)/2 + 1 = 112.5 -> floor 112
    (56, 1, 1, 0, 56),
])
def test_conv_out_shape_floor(H, R, s, p, expect):
    assert oracle.conv2d_out_shape(H, H, R, R, s, s, p, p) == (expect, expect)


def test_conv_out_shape_rejects_bad():
    with pytest.raises(ValueError):
        oracle.conv2d_out_shape(4, 4, 7, 7, 1, 1, 0, 0)  # kernel larger than padded input
    with pytest.raises(ValueError):
        oracle.conv2d_out_shape(4, 4, 3, 3, 0, 1, 0, 0)  # zero stride


# ---------------------------------------------------------------- closed forms
@pytest.mark.parametrize("stride,pad", [(1, 0), (1, 2), (2, 1), (4, 0), (3, 2)])
@pytest.mark.parametrize("r0,s0", [(0, 0), (1, 2), (2, 0)])
def test_conv_delta_kernel_is_shifted_sample(stride, pad, r0, s0):
    """w = delta(r0, s0) selects x[p*st - pad + r0, q*st - pad + s0] (0 outside): this
    tells cross-correlation from convolution (a flip would select R-1-r0)."""
    H, W, R, S = 11, 9, 3, 4
    x = _rand((2, 1, H, W), 1)
    w = np.zeros((1, 1, R, S), np.float32)
    w[0, 0, r0, s0] = 1.0
    y = oracle.conv2d_fwd(x, w, stride=(stride, stride), pad=(pad, pad))
    P, Q = y.shape[2:]
    for p in range(P):
        for q in range(Q):
            h, ww = p * stride - pad + r0, q * stride - pad + s0
            expect = x[:, 0, h, ww] if (0 <= h < H and 0 <= ww < W) else np.zeros(2, np.float32)
            np.testing.assert_array_equal(y[:, 0, p, q], expect)


@pytest.mark.parametrize("pad", [0, 1, 2])
def test_conv_constant_input_counts_taps(pad):
    """Constant input c0, all-ones weights: y = b + c0 * C * (#taps inside the image)."""
    C, H, W, R, S, c0, b = 3, 6, 5, 3, 3, 0.5, 0.25
    x = np.full((1, C, H, W), c0, np.float32)
    w = np.ones((2, C, R, S), np.float32)
    y = oracle.conv2d_fwd(x, w, np.array([b, -b], np.float32), pad=(pad, pad))
    P, Q = y.shape[2:]
    for p in range(P):
        rows = sum(1 for r in range(R) if 0 <= p - pad + r < H)
        for q in range(Q):
            cols = sum(1 for s in range(S) if 0 <= q - pad + s < W)
            assert y[0, 0, p, q] == np.float32(b + c0 * C * rows * cols)
            assert y[0, 1, p, q] == np.float32(-b + c0 * C * rows * cols)


def test_conv_1x1_identity_weights():
    x = _rand((2, 5, 4, 3), 2)
    w = np.eye(5, dtype=np.float32).reshape(5, 5, 1, 1)
    np.testing.assert_array_equal(oracle.conv2d_fwd(x, w), x)


# ---------------------------------------------------------------- invariants
def test_conv_linear_in_weights_and_input():
    x1, x2 = _rand((2, 4, 7, 7), 3), _rand((2, 4, 7, 7), 4)
    w1, w2 = _rand((6, 4, 3, 3), 5), _rand((6, 4, 3, 3), 6)
    a, b = 0.75, -1.5
    lhs = oracle.conv2d_fwd(x1, a * w1 + b * w2, pad=(1, 1)).astype(np.float64)
    rhs = (a * oracle.conv2d_fwd(x1, w1, pad=(1, 1)).astype(np.float64)
           + b * oracle.conv2d_fwd(x1, w2, pad=(1, 1)).astype(np.float64))
    np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-5)
    lhs = oracle.conv2d_fwd(a * x1 + b * x2, w1, pad=(1, 1)).astype(np.float64)
    rhs = (a * oracle.conv2d_fwd(x1, w1, pad=(1, 1)).astype(np.float64)
           + b * oracle.conv2d_fwd(x2, w1, pad=(1, 1)).astype(np.float64))
    np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-5)


def test_conv_grouped_is_concatenation():
    """Group g sees input channels [g*C/G, (g+1)*C/G) and produces outputs [g*K/G, ...)."""
    G, C, K = 3, 6, 9
    x = _rand((2, C, 8, 8), 7)
    w = _rand((K, C // G, 3, 3), 8)
    b = _rand((K,), 9)
    y = oracle.conv2d_fwd(x, w, b, stride=(2, 2), pad=(1, 1), groups=G)
    parts = [oracle.conv2d_fwd(x[:, g * 2:(g + 1) * 2], w[g * 3:(g + 1) * 3], b[g * 3:(g + 1) * 3],
                               stride=(2, 2), pad=(1, 1)) for g in range(G)]
    np.testing.assert_array_equal(y, np.concatenate(parts, axis=1))


def test_conv_relu_flag_is_relu_after():
    x, w, b = _rand((2, 3, 6, 6), 10), _rand((4, 3, 3, 3), 11), _rand((4,), 12)
    y = oracle.conv2d_fwd(x, w, b)
    np.testing.assert_array_equal(oracle.conv2d_fwd(x, w, b, relu=True), np.where(y > 0, y, 0))


# ---------------------------------------------------------------- library witness
@pytest.mark.parametrize("N,C,H,W,K,R,S,st,pd,G", [
    (2, 3, 17, 13, 5, 5, 3, 2, 2, 1),
    (1, 4, 9, 9, 6, 3, 3, 1, 1, 2),
    (3, 1, 12, 12, 4, 5, 5, 1, 0, 1),
    (1, 3, 23, 23, 8, 11, 11, 4, 0, 1),
    (2, 6, 7, 8, 6, 1, 1, 1, 0, 3),
])
def test_conv_matches_torch_float64(N, C, H, W, K, R, S, st, pd, G):
    x = _rand((N, C, H, W), 13)
    w = _rand((K, C // G, R, S), 14)
    b = _rand((K,), 15)
    y = oracle.conv2d_fwd(x, w, b, (st, st), (pd, pd), G)
    ref = F.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                   torch.from_numpy(b).double(), stride=st, padding=pd, groups=G).numpy()
    # the oracle rounds a double sum once to float: within half an ulp of the exact sum
    np.testing.assert_allclose(y, ref.astype(np.float32), rtol=1e-6, atol=1e-6)
    assert y.shape == ref.shape


# ---------------------------------------------------------------- fully connected
def test_fc_equals_conv_over_whole_image():
    """FC on the flattened NCHW tensor equals a conv whose kernel covers the image."""
    x = _rand((3, 4, 5, 6), 16)
    w = _rand((7, 4 * 5 * 6), 17)
    b = _rand((7,), 18)
    y_fc = oracle.fc_fwd(x.reshape(3, -1), w, b)
    y_conv = oracle.conv2d_fwd(x, w.reshape(7, 4, 5, 6), b)
    np.testing.assert_array_equal(y_fc, y_conv.reshape(3, 7))


def test_fc_identity_and_matmul_witness():
    x = _rand((5, 12), 19)
    np.testing.assert_array_equal(oracle.fc_fwd(x, np.eye(12, dtype=np.float32)), x)
    w, b = _rand((9, 12), 20), _rand((9,), 21)
    ref = x.astype(np.float64) @ w.astype(np.float64).T + b.astype(np.float64)
    np.testing.assert_allclose(oracle.fc_fwd(x, w, b), ref.astype(np.float32), rtol=1e-6, atol=1e-7)
    y = oracle.fc_fwd(x, w, b, relu=True)
    np.testing.assert_array_equal(y, np.maximum(oracle.fc_fwd(x, w, b), 0))


def test_fc_rejects_mismatched_features():
    with pytest.raises(ValueError):
        oracle.fc_fwd(_rand((2, 5), 0), _rand((3, 6), 1))


def test_conv_anisotropic_stride_pad_matches_torch():
    """Height and width strides/pads/kernels are independent."""
    x = _rand((2, 4, 15, 12), 22)
    w = _rand((6, 2, 3, 5), 23)
    b = _rand((6,), 24)
    y = oracle.conv2d_fwd(x, w, b, (2, 3), (1, 2), 2)
    ref = F.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                   torch.from_numpy(b).double(), stride=(2, 3), padding=(1, 2), groups=2).numpy()
    assert y.shape == ref.shape
    np.testing.assert_allclose(y, ref.astype(np.float32), rtol=1e-6, atol=1e-6)
