"""Pins of the oracle's pooling, LRN, ReLU and network composition (CPU only).

Each check is fixed by something other than the oracle: the hand-derived
fixtures under tests/golden/, the shape chain that the networks' FC input
sizes force, closed forms, invariants, or a torch CPU routine in float64.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from golden_io import load
from paper_1511_07376_amd import workloads as wl


def _rand(shape, seed, lo=-1.0, hi=1.0):
    return np.random.default_rng(seed).uniform(lo, hi, shape).astype(np.float32)


# ---------------------------------------------------------------- pool shapes
def test_pool_ceil_chain_forced_by_cifar_fc():
    """CIFAR-10 quick: FC 1024 -> 64 needs 64x4x4 after the third pooling.  Ceil mode
    gives 32 -> 16 -> 8 -> 4; floor mode would give 15 -> 7 -> 3 (64*3*3 = 576)."""
    h = 32
    for _ in range(3):
        h, _w = oracle.pool_out_shape(h, h, 3, 3, 2, 2, 0, 0, True)
    assert h == 4 and 64 * h * h == 1024
    h = 32
    for _ in range(3):
        h, _w = oracle.pool_out_shape(h, h, 3, 3, 2, 2, 0, 0, False)
    assert h == 3


@pytest.mark.parametrize("H,k,s,p,ceil,expect", [
    (55, 3, 2, 0, True, 27), (27, 3, 2, 0, True, 13), (13, 3, 2, 0, True, 6),   # AlexNet
    (24, 2, 2, 0, True, 12), (8, 2, 2, 0, True, 4),                             # LeNet
    (4, 3, 2, 1, True, 3),   # pad 1: no window dropped ((3-1)*2 = 4 < 5)
    (5, 2, 2, 1, True, 3),   # ceil gives 4; (4-1)*2 = 6 >= 5+1, so the last window is dropped
    (6, 3, 3, 1, True, 3),   # ceil((6+2-3)/3)+1 = 3; (3-1)*3 = 6 < 7 kept
    (5, 3, 3, 2, True, 3),   # ceil((5+4-3)/3)+1 = 3; (3-1)*3 = 6 >= 5+2? no -> 3
    (4, 2, 3, 1, True, 2),   # ceil((4+2-2)/3)+1 = 3; (3-1)*3 = 6 >= 4+1 -> dropped to 2
])
def test_pool_out_shape_cases(H, k, s, p, ceil, expect):
    assert oracle.pool_out_shape(H, H, k, k, s, s, p, p, ceil)[0] == expect


def test_pool_out_shape_matches_torch_ceil_rule():
    for H in range(3, 14):
        for k in (2, 3, 4):
            for s in (1, 2, 3):
                for p in range(0, k):
                    if H + 2 * p < k or p > k // 2:
                        continue  # torch additionally requires pad <= k/2
                    t = F.max_pool2d(torch.zeros(1, 1, H, H), k, s, p, ceil_mode=True)
                    assert oracle.pool_out_shape(H, H, k, k, s, s, p, p, True)[0] == t.shape[2]


def test_pool_rejects_pad_not_below_kernel():
    with pytest.raises(ValueError):
        oracle.pool_out_shape(8, 8, 2, 2, 2, 2, 2, 2, True)


# ---------------------------------------------------------------- pool fixtures
def test_pool_golden_ramp():
    g = load("pool_ramp4x4.txt")
    x = g["x"]
    np.testing.assert_array_equal(oracle.pool_fwd(x, "avg", (3, 3), (2, 2)), g["avg_p0"].astype(np.float32))
    y, i = oracle.pool_fwd(x, "max", (3, 3), (2, 2), with_index=True)
    np.testing.assert_array_equal(y, g["max_p0"].astype(np.float32))
    np.testing.assert_array_equal(i, g["idx_p0"].astype(np.int32))
    np.testing.assert_allclose(oracle.pool_fwd(x, "avg", (3, 3), (2, 2), (1, 1)),
                               g["avg_p1"].astype(np.float32), rtol=1e-7)
    y, i = oracle.pool_fwd(x, "max", (3, 3), (2, 2), (1, 1), with_index=True)
    np.testing.assert_array_equal(y, g["max_p1"].astype(np.float32))
    np.testing.assert_array_equal(i, g["idx_p1"].astype(np.int32))


def test_pool_ties_take_first_index():
    g = load("pool_ramp4x4.txt")
    _y, i = oracle.pool_fwd(np.zeros((1, 1, 4, 4), np.float32), "max", (2, 2), (2, 2), with_index=True)
    np.testing.assert_array_equal(i, g["idx_zero_k2s2"].astype(np.int32))
    x = np.zeros((1, 1, 4, 4), np.float32)
    x[0, 0, 0, 1] = x[0, 0, 1, 0] = 3.0   # two equal maxima in window (0, 0)
    _y, i = oracle.pool_fwd(x, "max", (2, 2), (2, 2), with_index=True)
    assert i[0, 0, 0, 0] == 1


# ---------------------------------------------------------------- pool witnesses / invariants
@pytest.mark.parametrize("H,W,k,s,p", [(9, 11, 3, 2, 0), (8, 8, 2, 2, 0), (10, 7, 3, 2, 1),
                                        (13, 13, 3, 2, 1), (7, 9, 4, 3, 2), (6, 6, 3, 1, 0)])
def test_pool_matches_torch(H, W, k, s, p):
    x = _rand((2, 3, H, W), 30)
    t = torch.from_numpy(x).double()
    y, i = oracle.pool_fwd(x, "max", (k, k), (s, s), (p, p), with_index=True)
    ty, ti = F.max_pool2d(t, k, s, p, ceil_mode=True, return_indices=True)
    np.testing.assert_array_equal(y, ty.float().numpy())
    np.testing.assert_array_equal(i, ti.numpy().astype(np.int32))  # distinct values: no ties
    ya = oracle.pool_fwd(x, "avg", (k, k), (s, s), (p, p))
    ta = F.avg_pool2d(t, k, s, p, ceil_mode=True, count_include_pad=True)
    np.testing.assert_allclose(ya, ta.float().numpy(), rtol=1e-6, atol=1e-7)


def test_pool_value_at_index_monotone_and_ordering():
    x = _rand((2, 4, 13, 13), 31)
    y, i = oracle.pool_fwd(x, "max", (3, 3), (2, 2), with_index=True)
    flat = x.reshape(2, 4, -1)
    np.testing.assert_array_equal(y, np.take_along_axis(flat, i.reshape(2, 4, -1), 2).reshape(y.shape))
    x2 = x + np.abs(_rand(x.shape, 32))   # x2 >= x elementwise
    assert np.all(oracle.pool_fwd(x2, "max", (3, 3), (2, 2)) >= y)
    assert np.all(oracle.pool_fwd(x2, "avg", (3, 3), (2, 2)) >= oracle.pool_fwd(x, "avg", (3, 3), (2, 2)))
    assert np.all(y >= oracle.pool_fwd(x, "avg", (3, 3), (2, 2)))
    c = np.full((1, 2, 9, 9), 0.375, np.float32)
    np.testing.assert_array_equal(oracle.pool_fwd(c, "avg", (3, 3), (2, 2)), 0.375)


def test_pool_then_relu_keeps_pre_relu_argmax():
    """Pooling+ReLU (CIFAR row 2): the index is the argmax before the ReLU."""
    x = -np.arange(1, 17, dtype=np.float32).reshape(1, 1, 4, 4)   # all negative, max at top-left
    x[0, 0, 1, 1] = -0.5
    y, i = oracle.pool_fwd(x, "max", (2, 2), (2, 2), relu=True, with_index=True)
    np.testing.assert_array_equal(y, 0.0)
    np.testing.assert_array_equal(i.ravel(), [5, 2, 8, 10])


# ---------------------------------------------------------------- LRN
def test_lrn_golden_single_channel():
    g = load("lrn_single_channel.txt")
    y = oracle.lrn_fwd(g["x"], int(g["size"]), g["alpha"], g["beta"], g["k"])
    np.testing.assert_allclose(y, g["y"].astype(np.float32), rtol=1e-6)
    assert abs(2.0 * 1.08 ** -0.75 - 1.887827) < 1e-6


@pytest.mark.parametrize("C,size,alpha,beta,k", [(7, 5, 1e-4, 0.75, 1.0), (16, 5, 0.5, 0.75, 2.0),
                                                  (5, 3, 1.0, 0.5, 1.0), (1, 5, 0.3, 0.75, 1.0),
                                                  (12, 7, 2.0, 1.0, 0.5)])
def test_lrn_matches_torch(C, size, alpha, beta, k):
    x = _rand((2, C, 5, 6), 40, -3, 3)
    y = oracle.lrn_fwd(x, size, alpha, beta, k)
    ref = F.local_response_norm(torch.from_numpy(x).double(), size, alpha, beta, k).numpy()
    np.testing.assert_allclose(y, ref.astype(np.float32), rtol=2e-6, atol=1e-7)


def test_lrn_special_cases():
    x = _rand((2, 6, 4, 4), 41, -2, 2)
    np.testing.assert_array_equal(oracle.lrn_fwd(x, 5, 0.0, 0.75, 1.0), x)   # alpha 0, k 1
    np.testing.assert_array_equal(oracle.lrn_fwd(np.zeros_like(x)), 0.0)
    np.testing.assert_array_equal(oracle.lrn_fwd(-x, 5, 0.5, 0.75, 1.0), -oracle.lrn_fwd(x, 5, 0.5, 0.75, 1.0))
    one = x[:, :1]   # C = 1: y = x * (k + alpha/size x^2)^-beta
    ref = one.astype(np.float64) * (1.0 + 0.5 / 5 * one.astype(np.float64) ** 2) ** -0.75
    np.testing.assert_allclose(oracle.lrn_fwd(one, 5, 0.5, 0.75, 1.0), ref.astype(np.float32), rtol=1e-6)
    with pytest.raises(ValueError):
        oracle.lrn_fwd(x, 4)   # even window sizes are rejected


# ---------------------------------------------------------------- ReLU
def test_relu_definition():
    x = np.array([-2.0, -0.0, 0.0, 1e-30, 3.5, -1e-30], np.float32)
    y = oracle.relu_fwd(x)
    np.testing.assert_array_equal(y, np.array([0, 0, 0, 1e-30, 3.5, 0], np.float32))
    assert not np.signbit(y[1])   # -0 maps to +0
    np.testing.assert_array_equal(oracle.relu_fwd(y), y)   # idempotent


# ---------------------------------------------------------------- networks
def _torch_net(net, x, params):
    """Independent witness: the same layer list through torch CPU ops in float64."""
    a = torch.from_numpy(x).double()
    for layer, pr in zip(net.layers, params):
        if layer.kind == "conv":
            a = F.conv2d(a, torch.from_numpy(pr[0]).double(), torch.from_numpy(pr[1]).double(),
                         stride=layer.stride, padding=layer.pad, groups=layer.groups)
        elif layer.kind == "fc":
            a = F.linear(a.reshape(a.shape[0], -1), torch.from_numpy(pr[0]).double(),
                         torch.from_numpy(pr[1]).double())
        elif layer.kind == "pool":
            fn = F.max_pool2d if layer.mode == "max" else F.avg_pool2d
            kw = {} if layer.mode == "max" else {"count_include_pad": True}
            a = fn(a, layer.kernel, layer.stride, layer.pad, ceil_mode=layer.ceil, **kw)
        elif layer.kind == "lrn":
            a = F.local_response_norm(a, layer.size, layer.alpha, layer.beta, layer.k)
        if layer.relu or layer.kind == "relu":
            a = torch.relu(a)
    return a.numpy()


@pytest.mark.parametrize("name,batch", [("lenet", 4), ("cifar_quick", 2), ("alexnet", 1)])
def test_net_matches_torch_float64(name, batch):
    net = wl.NETS[name]
    x = wl.make_input(net, batch, 0)
    params = wl.make_params(net, 0)
    y = oracle.net_fwd(net, x, params)
    ref = _torch_net(net, x, params)
    assert y.shape == ref.shape
    rel = np.linalg.norm(y - ref) / np.linalg.norm(ref)
    assert rel < 1e-5, rel


def test_net_shape_chain_matches_fc_inputs():
    """The stated FC input sizes (800, 1024, 9216) follow from the layer list."""
    for net in wl.NETS.values():
        c, h, w = net.input_chw
        for layer in net.layers:
            if layer.kind == "conv":
                h, w = oracle.conv2d_out_shape(h, w, *layer.kernel, *layer.stride, *layer.pad)
                c = layer.out_channels
            elif layer.kind == "pool":
                h, w = oracle.pool_out_shape(h, w, *layer.kernel, *layer.stride, *layer.pad, layer.ceil)
            elif layer.kind == "fc":
                assert c * h * w == layer.in_features, (net.name, c, h, w)
                c, h, w = layer.out_features, 1, 1


def test_pool_anisotropic_matches_torch():
    x = _rand((2, 3, 11, 14), 33)
    t = torch.from_numpy(x).double()
    y, i = oracle.pool_fwd(x, "max", (3, 2), (2, 3), (1, 0), with_index=True)
    ty, ti = F.max_pool2d(t, (3, 2), (2, 3), (1, 0), ceil_mode=True, return_indices=True)
    np.testing.assert_array_equal(y, ty.float().numpy())
    np.testing.assert_array_equal(i, ti.numpy().astype(np.int32))
    ya = oracle.pool_fwd(x, "avg", (3, 2), (2, 3), (1, 0))
    ta = F.avg_pool2d(t, (3, 2), (2, 3), (1, 0), ceil_mode=True, count_include_pad=True)
    np.testing.assert_allclose(ya, ta.float().numpy(), rtol=1e-6, atol=1e-7)
