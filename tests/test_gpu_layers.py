"""Layer parity: each libcnn entry point against the oracle on identical
seeded inputs (GPU).

Shapes: every layer of the LeNet-, CIFAR-10-quick- and AlexNet-shaped nets,
the single-layer conv sweep, and odd shapes with ragged tiles (M, N and the
reduction not multiples of any tile; C = 1 and 3; strides 2 to 4; pads 0 to
3; groups 1 to 3).  Where the full batch is too much for the oracle, the GPU
runs the full batch and the oracle a few sampled images of it (images are
independent, so each sampled image must match exactly as if run alone).
"""
import numpy as np
import pytest
import torch

import oracle
from conftest import to_dev, to_host
from paper_1511_07376_amd import workloads as wl
from parity import assert_elementwise_close, assert_gemm_close

pytestmark = pytest.mark.gpu


def _conv_case(gpu, N, C, H, W, K, R, S, st, pd, G, relu=True, bias=True, seed=0,
               sample=None, dist="normal", wstd=1.0):
    tag = f"conv N{N} C{C} {H}x{W} K{K} {R}x{S} s{st} p{pd} G{G} relu{int(relu)} seed{seed}"
    print(tag, flush=True)
    if dist == "normal":
        x = wl.normal((N, C, H, W), 1.0, seed, 0)
    else:
        x = wl.uniform01((N, C, H, W), seed, 0)
    w = wl.normal((K, C // G, R, S), wstd, seed, 1)
    b = wl.normal((K,), 1.0, seed, 2) if bias else None
    y = gpu.cnn_conv2d_fwd(to_dev(x), to_dev(w), to_dev(b) if bias else None, st, pd, G, relu)
    yg = to_host(y)
    rows = list(range(N)) if sample is None else sample
    ref = oracle.conv2d_fwd(x[rows], w, b, _pair(st), _pair(pd), G, relu)
    assert_gemm_close(yg[rows], ref, (C // G) * R * S, tag)


def _pair(v):
    return (v, v) if isinstance(v, int) else v


# ---------------------------------------------------------------- network layers
NET_CONVS = []
for _net in (wl.lenet, wl.cifar_quick, wl.alexnet):
    _c, _h, _w = _net.input_chw
    for _layer in _net.layers:
        if _layer.kind == "conv":
            NET_CONVS.append((_net.name, _layer, _c, _h, _w))
            _h, _w = oracle.conv2d_out_shape(_h, _w, *_layer.kernel, *_layer.stride, *_layer.pad)
            _c = _layer.out_channels
        elif _layer.kind == "pool":
            _h, _w = oracle.pool_out_shape(_h, _w, *_layer.kernel, *_layer.stride, *_layer.pad, _layer.ceil)


@pytest.mark.parametrize("case", NET_CONVS, ids=lambda c: f"{c[0]}-{c[1].in_channels}to{c[1].out_channels}")
def test_conv_net_layers(gpu, case):
    name, layer, C, H, W = case
    N = {"lenet": 16, "cifar_quick": 32, "alexnet": 3}[name]
    _conv_case(gpu, N, C, H, W, layer.out_channels, *layer.kernel, layer.stride, layer.pad,
               layer.groups, relu=layer.relu, seed=1, dist="uniform", wstd=0.05)


@pytest.mark.parametrize("case", [c for c in NET_CONVS if c[0] == "alexnet"],
                         ids=lambda c: f"alexnet-b64-{c[1].in_channels}to{c[1].out_channels}")
def test_conv_alexnet_batch64_sampled(gpu, case):
    _name, layer, C, H, W = case
    _conv_case(gpu, 64, C, H, W, layer.out_channels, *layer.kernel, layer.stride, layer.pad,
               layer.groups, relu=layer.relu, seed=2, sample=[0, 37, 63], dist="uniform", wstd=0.01)


@pytest.mark.parametrize("shape", wl.SWEEP_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv_sweep_batch1(gpu, shape):
    C, H, W, K, R, S, st, pd = shape
    _conv_case(gpu, 1, C, H, W, K, R, S, st, pd, 1, seed=3)


@pytest.mark.parametrize("shape", wl.SWEEP_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv_sweep_batch16_sampled(gpu, shape):
    C, H, W, K, R, S, st, pd = shape
    _conv_case(gpu, 16, C, H, W, K, R, S, st, pd, 1, seed=6, sample=[0, 7, 15])


@pytest.mark.parametrize("shape", wl.SWEEP_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv_sweep_batch64_sampled(gpu, shape):
    C, H, W, K, R, S, st, pd = shape
    _conv_case(gpu, 64, C, H, W, K, R, S, st, pd, 1, seed=4, sample=[0, 63])


@pytest.mark.parametrize("batch", [16, 64])
@pytest.mark.parametrize("shape", wl.SWEEP_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv_sweep_every_config(gpu, shape, batch):
    """Every tile configuration on each conv-sweep shape at batches 16 and 64
    (the benchmark's sweep auto-tunes, so any of them may be the one timed);
    sampled images."""
    C, H, W, K, R, S, st, pd = shape
    x = wl.normal((batch, C, H, W), 1.0, 24, 0)
    w = wl.normal((K, C, R, S), 1.0, 24, 1)
    b = wl.normal((K,), 1.0, 24, 2)
    rows = [0, batch - 1]
    ref = oracle.conv2d_fwd(x[rows], w, b, (st, st), (pd, pd), 1, True)
    xd, wd, bd = to_dev(x), to_dev(w), to_dev(b)
    for cfg in range(gpu.cnn_conv2d_num_configs()):
        print(f"sweep {shape} N{batch} config {cfg}", flush=True)
        y = gpu.cnn_conv2d_fwd(xd, wd, bd, st, pd, 1, True, config=cfg)
        torch.cuda.synchronize()
        assert_gemm_close(y[rows].cpu().numpy(), ref, C * R * S, f"config {cfg}")
        del y


# The five AlexNet conv layers at batch 64 as the network runs them: conv2
# and conv3 read planes that the LRN + pooling kernel before them wrote
# inside a zero border of their padding width, and run unpadded on the
# bordered (H + 2p) x (W + 2p) planes.  (N, C, H, W, K, R, S, stride, pad, G)
ALEXNET_B64_AS_RUN = [
    (64, 3, 227, 227, 96, 11, 11, 4, 0, 1),
    (64, 96, 31, 31, 256, 5, 5, 1, 0, 2),
    (64, 256, 15, 15, 384, 3, 3, 1, 0, 1),
    (64, 384, 13, 13, 384, 3, 3, 1, 1, 2),
    (64, 384, 13, 13, 256, 3, 3, 1, 1, 2),
]


@pytest.mark.parametrize("shape", ALEXNET_B64_AS_RUN, ids=[f"conv{i + 1}" for i in range(5)])
def test_conv_alexnet_b64_every_config(gpu, shape):
    """Every tile configuration (and the heuristic) on each AlexNet batch-64
    conv shape, so that whichever configuration the auto-tuner keeps for the
    benchmark has been checked at that exact shape; sampled images."""
    N, C, H, W, K, R, S, st, pd, G = shape
    x = wl.normal((N, C, H, W), 1.0, 23, 0)
    w = wl.normal((K, C // G, R, S), 1.0, 23, 1)
    b = wl.normal((K,), 1.0, 23, 2)
    rows = [0, 31, 63]
    ref = oracle.conv2d_fwd(x[rows], w, b, (st, st), (pd, pd), G, True)
    xd, wd, bd = to_dev(x), to_dev(w), to_dev(b)
    for cfg in range(-1, gpu.cnn_conv2d_num_configs()):
        print(f"alexnet b64 conv config {cfg} ({gpu.cnn_conv2d_config_name(cfg)}) shape {shape}", flush=True)
        y = gpu.cnn_conv2d_fwd(xd, wd, bd, st, pd, G, True, config=cfg)
        assert_gemm_close(to_host(y)[rows], ref, (C // G) * R * S, f"config {cfg}")


# ---------------------------------------------------------------- odd shapes
ODD = [
    # N, C, H, W, K, R, S, stride, pad, G, relu, bias
    (1, 1, 7, 7, 1, 3, 3, 1, 0, 1, False, True),
    (3, 5, 13, 17, 7, 3, 2, (2, 1), (1, 0), 1, True, True),
    (2, 6, 9, 11, 10, 5, 5, 1, 2, 2, True, False),
    (2, 1, 30, 30, 33, 5, 5, 1, 0, 1, True, True),
    (1, 3, 37, 41, 65, 11, 11, 4, 0, 1, True, True),
    (2, 16, 10, 10, 129, 3, 3, 1, 1, 1, False, True),
    (2, 48, 6, 6, 96, 3, 3, 1, 1, 3, True, True),
    (1, 12, 8, 8, 300, 1, 1, 1, 0, 2, True, True),
    (5, 7, 5, 5, 3, 5, 5, 1, 0, 1, False, True),
    (1, 4, 9, 9, 8, 3, 3, 3, 3, 1, True, True),
    (2, 3, 19, 23, 97, 7, 7, 2, 3, 1, True, True),
    (1, 64, 4, 4, 33, 4, 4, 1, 0, 1, False, True),
    (2, 20, 12, 12, 50, 5, 5, 1, 0, 1, False, True),
    (1, 256, 3, 3, 200, 3, 3, 1, 1, 1, True, True),
]


@pytest.mark.parametrize("case", ODD, ids=[f"odd{i}" for i in range(len(ODD))])
def test_conv_odd_shapes(gpu, case):
    N, C, H, W, K, R, S, st, pd, G, relu, bias = case
    _conv_case(gpu, N, C, H, W, K, R, S, st, pd, G, relu, bias, seed=5)


def test_conv_empty_batch(gpu):
    x = torch.empty((0, 3, 8, 8), device="cuda")
    w = torch.ones((4, 3, 3, 3), device="cuda")
    y = gpu.cnn_conv2d_fwd(x, w)
    assert y.shape == (0, 4, 6, 6)


def test_conv_does_not_write_past_output(gpu):
    x = wl.normal((2, 8, 11, 11), 1.0, 6, 0)
    w = wl.normal((13, 8, 3, 3), 1.0, 6, 1)
    P, Q = oracle.conv2d_out_shape(11, 11, 3, 3, 1, 1, 1, 1)
    n = 2 * 13 * P * Q
    buf = torch.full((n + 4096,), 12345.0, device="cuda")
    gpu.cnn_conv2d_fwd(to_dev(x), to_dev(w), None, 1, 1, 1, False, y=buf[:n].view(2, 13, P, Q))
    out = to_host(buf)
    assert np.all(out[n:] == 12345.0)
    assert_gemm_close(out[:n].reshape(2, 13, P, Q), oracle.conv2d_fwd(x, w, None, (1, 1), (1, 1)),
                      72, "canary conv")


# ---------------------------------------------------------------- fully connected
FC_CASES = [
    # N, I, O, relu, sample
    (16, 800, 500, True, None), (16, 500, 10, False, None),          # LeNet
    (32, 1024, 64, False, None), (32, 64, 10, False, None),          # CIFAR-10 quick
    (16, 9216, 4096, True, None), (16, 4096, 4096, True, None), (16, 4096, 1000, False, None),
    (64, 9216, 4096, True, [0, 31, 63]), (64, 4096, 1000, False, None),
    (256, 9216, 4096, True, [0, 100, 255]), (256, 4096, 4096, True, [1, 254]),
    (1, 37, 3, False, None), (5, 1001, 31, True, None), (33, 129, 129, False, None),
    (65, 260, 7, True, None), (130, 64, 300, False, None), (3, 4, 1, True, None),
    # batches up to 64 with inputs a multiple of 4, split and unsplit; the
    # direct kernel's built-in cases (at most 32 images, 4096 inputs and 2048
    # features): one and two waves' runs of the reduction, a ragged 32-feature
    # block
    (48, 512, 300, True, None), (20, 3072, 4100, True, [0, 7, 19]), (64, 96, 17, False, None),
    (16, 4096, 1000, True, None), (7, 64, 33, False, None), (32, 2048, 2000, True, [0, 31]),
    # batches of 1 and 2: the matrix-vector kernel (128-bit and 32-bit loads,
    # 4-row and 1-row workgroups, a ragged last workgroup); 3 and 4 images on
    # the matrix cores next to them
    (1, 9216, 4096, True, None), (2, 4096, 1000, False, None), (2, 4100, 4098, True, [0, 1]),
    (1, 4096, 4101, False, None), (4, 1024, 33, True, None), (4, 100, 7, False, None),
    (2, 1001, 13, True, None),
]


@pytest.mark.parametrize("case", FC_CASES, ids=[f"fc{c[0]}x{c[1]}to{c[2]}" for c in FC_CASES])
def test_fc(gpu, case):
    N, I, O, relu, sample = case
    tag = f"fc N{N} I{I} O{O} relu{int(relu)}"
    print(tag, flush=True)
    x = wl.uniform01((N, I), 7, 0)
    w = wl.normal((O, I), 0.05, 7, 1)
    b = wl.normal((O,), 0.01, 7, 2)
    yg = to_host(gpu.cnn_fc_fwd(to_dev(x), to_dev(w), to_dev(b), relu))
    rows = list(range(N)) if sample is None else sample
    assert_gemm_close(yg[rows], oracle.fc_fwd(x[rows], w, b, relu), I, tag)


FC_CFG_CASES = [
    # N, I, O, relu, sampled rows: AlexNet's fc6-fc8 at batches 16 and 64,
    # ragged batches, features and reductions (multiples of 4 and not), a
    # reduction shorter than one 32-tap chunk, batches above 64
    (64, 9216, 4096, True, [0, 31, 32, 63]), (64, 4096, 4096, True, [1, 62]), (64, 4096, 1000, False, None),
    (16, 9216, 4096, True, [0, 15]), (16, 4096, 1000, False, None),
    (33, 1000, 33, True, None), (5, 4100, 70, False, None), (64, 12, 5, True, None),
    (2, 4096, 300, False, None), (1, 36, 1, True, None), (31, 1001, 31, True, None), (70, 256, 64, False, None),
]


@pytest.mark.parametrize("case", FC_CFG_CASES, ids=[f"fc{c[0]}x{c[1]}to{c[2]}" for c in FC_CFG_CASES])
def test_fc_every_config(gpu, case):
    """Every FC configuration on the shape; a configuration that does not take
    it (batch above its limit, a reduction not a multiple of 4 for the
    128-bit-load ones) must say so with CNN_ERR_UNSUPPORTED."""
    N, I, O, relu, sample = case
    x = wl.uniform01((N, I), 17, 0)
    w = wl.normal((O, I), 0.05, 17, 1)
    b = wl.normal((O,), 0.01, 17, 2)
    rows = list(range(N)) if sample is None else sample
    ref = oracle.fc_fwd(x[rows], w, b, relu)
    xd, wd, bd = to_dev(x), to_dev(w), to_dev(b)
    ran = 0
    for cfg in range(gpu.cnn_fc_num_configs()):
        tag = f"fc N{N} I{I} O{O} relu{int(relu)} config {cfg} ({gpu.cnn_fc_config_name(cfg)})"
        print(tag, flush=True)
        y = torch.full((N, O), float("nan"), device="cuda")
        rc = gpu.lib.cnn_fc_fwd_config(xd.data_ptr(), N, I, wd.data_ptr(), bd.data_ptr(), O, int(relu),
                                       y.data_ptr(), cfg, torch.cuda.current_stream().cuda_stream)
        if rc == gpu.CNN_ERR_UNSUPPORTED:
            continue
        assert rc == 0, gpu.cnn_last_error()
        assert_gemm_close(to_host(y)[rows], ref, I, tag)
        ran += 1
    assert ran >= 2


@pytest.mark.parametrize("N", [7, 2])
def test_fc_unaligned_and_no_bias(gpu, N):
    x = wl.normal((N * 96 + 1,), 1.0, 8, 0)
    w = wl.normal((40, 96), 1.0, 8, 1)
    xd = to_dev(x)[1:]                     # 4-byte offset: not 16-byte aligned
    ref_in = x[1:].reshape(N, 96)
    # unaligned pointer through the raw ABI
    y = torch.empty((N, 40), device="cuda")
    rc = gpu.lib.cnn_fc_fwd(xd.data_ptr(), N, 96, to_dev(w).data_ptr(), None, 40, 0, y.data_ptr(),
                            torch.cuda.current_stream().cuda_stream)
    assert rc == 0, gpu.cnn_last_error()
    assert_gemm_close(to_host(y), oracle.fc_fwd(ref_in, w, None), 96, f"fc unaligned N{N}")


# ---------------------------------------------------------------- pooling
POOL_CASES = [
    # N, C, H, W, mode, k, s, p, relu
    (16, 20, 24, 24, "max", 2, 2, 0, False), (16, 50, 8, 8, "max", 2, 2, 0, False),   # LeNet
    (32, 32, 32, 32, "max", 3, 2, 0, True), (32, 32, 16, 16, "avg", 3, 2, 0, False),  # CIFAR
    (32, 64, 8, 8, "avg", 3, 2, 0, False),
    (4, 96, 55, 55, "max", 3, 2, 0, False), (4, 256, 27, 27, "max", 3, 2, 0, False),  # AlexNet
    (4, 256, 13, 13, "max", 3, 2, 0, False),
    (2, 3, 10, 7, "max", 3, 2, 1, False), (2, 3, 10, 7, "avg", 3, 2, 1, True),
    (1, 5, 9, 9, "max", (3, 2), (2, 3), (1, 0), True), (1, 5, 9, 9, "avg", (3, 2), (2, 3), (1, 0), False),
    (3, 2, 7, 9, "max", 4, 3, 2, False), (3, 2, 7, 9, "avg", 4, 3, 2, False),
    (1, 1, 1, 1, "max", 1, 1, 0, False), (2, 4, 5, 5, "avg", 5, 1, 0, False),
    # planes of more than 48 KiB (pooled straight from memory, not staged in LDS)
    (1, 2, 130, 120, "max", 3, 2, 1, False), (1, 2, 130, 120, "avg", 3, 2, 1, True),
    (3, 5, 57, 57, "max", 3, 3, 0, False),
]


@pytest.mark.parametrize("case", POOL_CASES, ids=[f"pool{i}" for i in range(len(POOL_CASES))])
def test_pool(gpu, case):
    N, C, H, W, mode, k, s, p, relu = case
    tag = f"pool N{N} C{C} {H}x{W} {mode} k{k} s{s} p{p} relu{int(relu)}"
    print(tag, flush=True)
    x = wl.normal((N, C, H, W), 1.0, 9, 0)
    k, s, p = _pair(k), _pair(s), _pair(p)
    if mode == "max":
        yg, ig = gpu.cnn_pool_fwd(to_dev(x), "max", k, s, p, True, relu, with_index=True)
        yr, ir = oracle.pool_fwd(x, "max", k, s, p, True, relu, with_index=True)
        np.testing.assert_array_equal(to_host(yg), yr, err_msg=tag)
        np.testing.assert_array_equal(to_host(ig), ir, err_msg=tag)
    else:
        yg = gpu.cnn_pool_fwd(to_dev(x), "avg", k, s, p, True, relu)
        yr = oracle.pool_fwd(x, "avg", k, s, p, True, relu)
        assert_elementwise_close(to_host(yg), yr, np.abs(x).max(), tag)


def test_maxpool_ties_and_relu_window(gpu):
    """Many equal values (quantised, ReLU'd input): the first maximum in row-major order."""
    x = np.maximum(np.round(wl.normal((4, 8, 27, 27), 1.0, 10, 0) * 2) / 2, 0).astype(np.float32)
    yg, ig = gpu.cnn_pool_fwd(to_dev(x), "max", 3, 2, 0, True, False, with_index=True)
    yr, ir = oracle.pool_fwd(x, "max", (3, 3), (2, 2), (0, 0), True, False, with_index=True)
    np.testing.assert_array_equal(to_host(yg), yr)
    np.testing.assert_array_equal(to_host(ig), ir)
    # all-negative windows with the ReLU after pooling keep the pre-ReLU argmax
    xn = -np.abs(wl.normal((2, 3, 8, 8), 1.0, 11, 0))
    yg, ig = gpu.cnn_pool_fwd(to_dev(xn), "max", 2, 2, 0, True, True, with_index=True)
    yr, ir = oracle.pool_fwd(xn, "max", (2, 2), (2, 2), (0, 0), True, True, with_index=True)
    np.testing.assert_array_equal(to_host(yg), yr)
    np.testing.assert_array_equal(to_host(ig), ir)


# ---------------------------------------------------------------- LRN
LRN_CASES = [
    # N, C, H, W, size, alpha, beta, k
    (2, 96, 55, 55, 5, 1e-4, 0.75, 1.0), (2, 256, 27, 27, 5, 1e-4, 0.75, 1.0),   # AlexNet
    (3, 7, 5, 6, 5, 0.5, 0.75, 2.0), (2, 1, 4, 4, 5, 0.3, 0.75, 1.0), (2, 9, 3, 5, 3, 1.0, 0.5, 1.0),
    (1, 12, 4, 4, 1, 2.0, 0.75, 1.0), (1, 20, 3, 3, 9, 1.0, 0.75, 1.0), (1, 30, 3, 3, 11, 2.0, 1.0, 0.5),
    (2, 3, 2, 2, 7, 1.0, 0.75, 1.0),
]


@pytest.mark.parametrize("case", LRN_CASES, ids=[f"lrn{i}" for i in range(len(LRN_CASES))])
def test_lrn(gpu, case):
    N, C, H, W, size, alpha, beta, k = case
    tag = f"lrn N{N} C{C} {H}x{W} size{size} a{alpha} b{beta} k{k}"
    print(tag, flush=True)
    x = wl.normal((N, C, H, W), 3.0, 12, 0)
    yg = to_host(gpu.cnn_lrn_fwd(to_dev(x), size, alpha, beta, k))
    assert_elementwise_close(yg, oracle.lrn_fwd(x, size, alpha, beta, k), np.abs(x).max(), tag)


# ---------------------------------------------------------------- ReLU
@pytest.mark.parametrize("n", [0, 1, 3, 4, 5, 1023, (1 << 20) + 3])
def test_relu(gpu, n):
    x = wl.normal((n,), 1.0, 13, 0)
    x[: min(n, 3)] = np.array([-0.0, 0.0, -1e-30], np.float32)[: min(n, 3)]
    yg = to_host(gpu.cnn_relu_fwd(to_dev(x)))
    np.testing.assert_array_equal(yg, oracle.relu_fwd(x))
    assert not np.any(np.signbit(yg))


def test_relu_in_place_and_unaligned(gpu):
    x = wl.normal((4099,), 1.0, 14, 0)
    xd = to_dev(x)
    gpu.cnn_relu_fwd(xd, y=xd)
    np.testing.assert_array_equal(to_host(xd), oracle.relu_fwd(x))
    xd = to_dev(x)
    sub = xd[1:]   # 4-byte offset
    gpu.cnn_relu_fwd(sub, y=sub)
    out = to_host(xd)
    assert out[0] == x[0]
    np.testing.assert_array_equal(out[1:], oracle.relu_fwd(x[1:]))


# ---------------------------------------------------------------- errors through the binding
def test_binding_errors(gpu):
    x = torch.zeros((1, 3, 8, 8), device="cuda")
    with pytest.raises(gpu.CnnError) as e:
        gpu.cnn_conv2d_fwd(x, torch.zeros((4, 1, 3, 3), device="cuda"), groups=2)
    assert e.value.status == gpu.CNN_ERR_INVALID
    with pytest.raises(TypeError):
        gpu.cnn_relu_fwd(torch.zeros(4))   # host tensor
    with pytest.raises(TypeError):
        gpu.cnn_relu_fwd(torch.zeros(4, device="cuda", dtype=torch.float64))
    with pytest.raises(gpu.CnnError):
        gpu.cnn_lrn_fwd(x, size=4)


# ---------------------------------------------------------------- every tile configuration
CFG_SHAPES = [
    # N, C, H, W, K, R, S, stride, pad, G
    # reductions divisible by 4 (128-bit weight loads) and not (32-bit loads);
    # gather modes: padded filters of <= 31 taps (mask), unpadded (no-pad),
    # unpadded with a stride (strided), padded with a stride (strided mask,
    # 7x7 and 5x5), padded stride-1 7x7 and a reduction too long for the LDS
    # tap table (scalar)
    (2, 8, 12, 13, 70, 3, 3, 1, 1, 1),
    (2, 32, 9, 9, 130, 1, 1, 1, 0, 2),
    (2, 3, 23, 21, 40, 7, 7, 2, 3, 1),
    (1, 1024, 5, 6, 36, 3, 3, 1, 1, 1),
    (2, 5, 13, 11, 70, 3, 3, 1, 1, 1),
    (3, 6, 17, 19, 130, 5, 5, 2, 2, 2),
    (1, 3, 31, 29, 97, 11, 11, 4, 0, 1),
    (2, 4, 19, 23, 40, 3, 3, 2, 0, 1),     # strided gathers: stride 2, 128-bit weight loads
    (1, 6, 40, 37, 70, 5, 5, 3, 0, 2),     # stride 3, two groups, ragged pixel tiles
    # few output tiles: the reduction is split across workgroups (mask, no-pad
    # and scalar gathers; chunks that start inside a filter; a ragged last
    # chunk with 32-bit weight loads and two groups)
    (1, 256, 7, 7, 64, 3, 3, 1, 1, 1),
    (1, 512, 6, 5, 40, 1, 1, 1, 0, 1),
    (1, 64, 9, 9, 20, 7, 7, 1, 3, 1),
    (1, 100, 5, 5, 30, 3, 3, 1, 1, 2),
    (1, 96, 15, 15, 40, 3, 3, 2, 0, 1),    # split reduction with the strided gather
    (1, 64, 17, 17, 40, 3, 3, 2, 1, 1),    # split reduction with the strided, padded gather
]


@pytest.mark.parametrize("shape", CFG_SHAPES, ids=[f"shape{i}" for i in range(len(CFG_SHAPES))])
def test_conv_every_config(gpu, shape):
    N, C, H, W, K, R, S, st, pd, G = shape
    x = wl.normal((N, C, H, W), 1.0, 20, 0)
    w = wl.normal((K, C // G, R, S), 1.0, 20, 1)
    b = wl.normal((K,), 1.0, 20, 2)
    ref = oracle.conv2d_fwd(x, w, b, (st, st), (pd, pd), G, True)
    xd, wd, bd = to_dev(x), to_dev(w), to_dev(b)
    for cfg in range(-1, gpu.cnn_conv2d_num_configs()):
        print(f"conv config {cfg} ({gpu.cnn_conv2d_config_name(cfg)}) shape {shape}", flush=True)
        y = gpu.cnn_conv2d_fwd(xd, wd, bd, st, pd, G, True, config=cfg)
        assert_gemm_close(to_host(y), ref, (C // G) * R * S, f"config {cfg}")


def test_autotune_records_and_reuses(gpu):
    shape = (4, 16, 14, 14, 96, 3, 3, 1, 1, 1)
    N, C, H, W, K, R, S, st, pd, G = shape
    x = wl.normal((N, C, H, W), 1.0, 21, 0)
    w = wl.normal((K, C, R, S), 1.0, 21, 1)
    ref = oracle.conv2d_fwd(x, w, None, (st, st), (pd, pd), G, False)
    gpu.cnn_tuning_clear()
    gpu.cnn_set_autotune(True)
    try:
        y = gpu.cnn_conv2d_fwd(to_dev(x), to_dev(w), None, st, pd, G, False)
        assert_gemm_close(to_host(y), ref, C * R * S, "autotuned call")
    finally:
        gpu.cnn_set_autotune(False)
    text = gpu.cnn_tuning_export()
    lines = [l for l in text.splitlines() if l.startswith("4 16 14 14 96 3 3 1 1 1 1 1 ")]
    assert len(lines) == 1, text
    cfg = int(lines[0].split()[-1])
    assert 0 <= cfg < gpu.cnn_conv2d_num_configs()
    y = gpu.cnn_conv2d_fwd(to_dev(x), to_dev(w), None, st, pd, G, False)   # uses the record
    assert_gemm_close(to_host(y), ref, C * R * S, "tuned record")
    gpu.cnn_tuning_clear()


@pytest.mark.parametrize("bias,relu", [(False, False), (True, False), (False, True)])
def test_conv_split_reduction_bias_relu_and_bounds(gpu, bias, relu):
    """A batch of one image with a long reduction takes the split path (output
    pre-filled with the bias, partial tiles added atomically, ReLU after):
    every combination of bias and ReLU matches, and nothing past the output
    is written."""
    N, C, H, W, K = 1, 384, 6, 6, 50
    x = wl.normal((N, C, H, W), 1.0, 21, 0)
    w = wl.normal((K, C, 3, 3), 1.0, 21, 1)
    b = wl.normal((K,), 1.0, 21, 2) if bias else None
    n = N * K * H * W
    for cfg in (-1, 2, 9, 14):
        print(f"split conv config {cfg} bias{int(bias)} relu{int(relu)}", flush=True)
        buf = torch.full((n + 4096,), -321.0, device="cuda")
        gpu.cnn_conv2d_fwd(to_dev(x), to_dev(w), to_dev(b) if bias else None, 1, 1, 1, relu,
                           y=buf[:n].view(N, K, H, W), config=cfg)
        out = to_host(buf)
        assert np.all(out[n:] == -321.0)
        ref = oracle.conv2d_fwd(x, w, b, (1, 1), (1, 1), 1, relu)
        assert_gemm_close(out[:n].reshape(N, K, H, W), ref, C * 9, f"split config {cfg}")


# ---------------------------------------------------------------- softmax
def _softmax_rtol(x, hw):
    """Per-element relative error bound of the GPU softmax against the double
    oracle: the shifted argument x - m rounded once (|x - m| ulps of 2^-24 in
    the exponential), exp itself (1 ulp), the sum of C terms (C/64 serial adds
    per lane plus 6 tree levels across the wave for HW = 1; C serial adds per
    thread otherwise) and one division; doubled as margin."""
    C = x.shape[1]
    span = float(np.max(np.max(x, axis=1, keepdims=True) - x)) if x.size else 0.0
    adds = C / 64 + 6 if hw == 1 else C
    return 2 * (span + adds + 2) * 2.0 ** -24


@pytest.mark.parametrize("shape", [(1, 1), (3, 10), (64, 1000), (2, 63), (2, 64), (2, 65), (5, 4097),
                                   (257, 7), (2, 3, 5, 7), (1, 21, 13, 13), (3, 1, 4, 4), (2, 1000, 1, 3)],
                         ids=lambda s: "x".join(map(str, s)))
def test_softmax(gpu, shape):
    print(f"softmax {shape}", flush=True)
    x = wl.normal(shape, 3.0, 22, 0)
    ref = oracle.softmax_fwd(x)
    y = to_host(gpu.cnn_softmax_fwd(to_dev(x)))
    hw = int(np.prod(shape[2:])) if len(shape) > 2 else 1
    np.testing.assert_allclose(y, ref, rtol=_softmax_rtol(x, hw), atol=1e-37)


def test_softmax_in_place_large_values_and_empty(gpu):
    x = np.array([[1000.0, 999.0, 998.0, -1000.0], [5.0, 5.0, 5.0, 5.0], [88.0, -88.0, 0.0, 1.0]],
                 dtype=np.float32)
    xd = to_dev(x)
    gpu.cnn_softmax_fwd(xd, y=xd)
    np.testing.assert_allclose(to_host(xd), oracle.softmax_fwd(x), rtol=_softmax_rtol(x, 1), atol=1e-37)
    assert np.all(to_host(xd)[1] == np.float32(0.25))
    x4 = wl.normal((2, 5, 3, 3), 2.0, 23, 0)
    xd = to_dev(x4)
    gpu.cnn_softmax_fwd(xd, y=xd)
    np.testing.assert_allclose(to_host(xd), oracle.softmax_fwd(x4), rtol=_softmax_rtol(x4, 9), atol=1e-37)
    assert gpu.cnn_softmax_fwd(torch.empty((0, 10), device="cuda")).shape == (0, 10)


# ---------------------------------------------------------------- random shapes
def _random_conv(seed):
    """A seeded random convolution: rectangular filters up to 7x7, strides
    and paddings per axis, groups, a tile configuration drawn from all of
    them (or the heuristic), batches that split or not."""
    rng = np.random.default_rng(9000 + seed)
    G = int(rng.choice([1, 1, 1, 2, 3, 4]))
    C = G * int(rng.integers(1, 17))
    K = G * int(rng.integers(1, 49))
    R, S = (int(v) for v in rng.integers(1, 8, size=2))
    sh, sw = (int(v) for v in rng.integers(1, 4, size=2))
    ph, pw = int(rng.integers(0, R)), int(rng.integers(0, S))
    H = int(rng.integers(max(1, R - 2 * ph), 33))
    W = int(rng.integers(max(1, S - 2 * pw), 33))
    N = int(rng.choice([1, 2, 3, 5, 9]))
    return N, C, H, W, K, R, S, (sh, sw), (ph, pw), G


@pytest.mark.parametrize("seed", range(48))
def test_conv_random_shapes(gpu, seed):
    N, C, H, W, K, R, S, st, pd, G = _random_conv(seed)
    cfg = int(np.random.default_rng(seed).integers(-1, gpu.cnn_conv2d_num_configs()))
    tag = f"random conv {seed}: N{N} C{C} {H}x{W} K{K} {R}x{S} s{st} p{pd} G{G} cfg{cfg}"
    print(tag, flush=True)
    x = wl.normal((N, C, H, W), 1.0, 40 + seed, 0)
    w = wl.normal((K, C // G, R, S), 1.0, 40 + seed, 1)
    b = wl.normal((K,), 1.0, 40 + seed, 2)
    y = gpu.cnn_conv2d_fwd(to_dev(x), to_dev(w), to_dev(b), st, pd, G, True, config=cfg)
    ref = oracle.conv2d_fwd(x, w, b, st, pd, G, True)
    assert_gemm_close(to_host(y), ref, (C // G) * R * S, tag)



def _random_pool(seed):
    """Seeded random pooling: windows up to 5x5 per axis, strides, paddings
    below the window, ceil or floor, planes small enough to stage in LDS and
    (one case in four) too large for it."""
    rng = np.random.default_rng(9500 + seed)
    kh, kw = (int(v) for v in rng.integers(1, 6, size=2))
    sh, sw = (int(v) for v in rng.integers(1, 5, size=2))
    ph, pw = int(rng.integers(0, kh)), int(rng.integers(0, kw))
    big = seed % 4 == 3
    H = int(rng.integers(max(1, kh - 2 * ph), 90 if big else 40))
    W = int(rng.integers(max(1, kw - 2 * pw), 90 if big else 40))
    if big:
        H, W = max(H, 66), max(W, 66)  # planes above 16 KiB
    N, C = int(rng.integers(1, 4)), int(rng.integers(1, 20))
    mode = "max" if seed % 2 == 0 else "avg"
    return N, C, H, W, mode, (kh, kw), (sh, sw), (ph, pw), bool(rng.integers(0, 2)), bool(seed % 3 == 1)


@pytest.mark.parametrize("seed", range(40))
def test_pool_random_shapes(gpu, seed):
    N, C, H, W, mode, k, s, p, ceil, relu = _random_pool(seed)
    tag = f"random pool {seed}: N{N} C{C} {H}x{W} {mode} k{k} s{s} p{p} ceil{int(ceil)} relu{int(relu)}"
    print(tag, flush=True)
    x = wl.normal((N, C, H, W), 1.0, 60 + seed, 0)
    if mode == "max":
        yg, ig = gpu.cnn_pool_fwd(to_dev(x), "max", k, s, p, ceil, relu, with_index=True)
        yr, ir = oracle.pool_fwd(x, "max", k, s, p, ceil, relu, with_index=True)
        np.testing.assert_array_equal(to_host(yg), yr, err_msg=tag)
        np.testing.assert_array_equal(to_host(ig), ir, err_msg=tag)
    else:
        yg = gpu.cnn_pool_fwd(to_dev(x), "avg", k, s, p, ceil, relu)
        yr = oracle.pool_fwd(x, "avg", k, s, p, ceil, relu)
        assert_elementwise_close(to_host(yg), yr, np.abs(x).max(), tag)


@pytest.mark.parametrize("seed", range(24))
def test_fc_random_shapes(gpu, seed):
    """Seeded random FC layers: batches from 1 (matrix-vector kernel) to 70,
    reductions that are and are not multiples of 4, with and without bias
    and ReLU."""
    rng = np.random.default_rng(9700 + seed)
    N = int(rng.choice([1, 2, 3, 7, 16, 31, 33, 64, 70]))
    I, O = int(rng.integers(1, 3000)), int(rng.integers(1, 700))
    relu, bias = bool(rng.integers(0, 2)), bool(rng.integers(0, 4))
    tag = f"random fc {seed}: N{N} I{I} O{O} relu{int(relu)} bias{int(bias)}"
    print(tag, flush=True)
    x = wl.normal((N, I), 1.0, 80 + seed, 0)
    w = wl.normal((O, I), 1.0, 80 + seed, 1)
    b = wl.normal((O,), 1.0, 80 + seed, 2) if bias else None
    yg = gpu.cnn_fc_fwd(to_dev(x), to_dev(w), to_dev(b) if bias else None, relu)
    assert_gemm_close(to_host(yg), oracle.fc_fwd(x, w, b, relu), I, tag)


@pytest.mark.parametrize("seed", range(16))
def test_lrn_random_shapes(gpu, seed):
    """Seeded random LRN: every odd size to 11 (the wide-window kernel above
    9), channel counts on both sides of the 32-channel chunk."""
    rng = np.random.default_rng(9900 + seed)
    size = int(rng.choice([1, 3, 5, 7, 9, 11]))
    N, C = int(rng.integers(1, 4)), int(rng.integers(1, 80))
    H, W = (int(v) for v in rng.integers(1, 30, size=2))
    alpha, beta, k = float(rng.uniform(1e-4, 0.1)), float(rng.uniform(0.5, 0.9)), float(rng.uniform(1.0, 2.0))
    tag = f"random lrn {seed}: N{N} C{C} {H}x{W} size{size} a{alpha:.4f} b{beta:.3f} k{k:.3f}"
    print(tag, flush=True)
    x = wl.normal((N, C, H, W), 3.0, 90 + seed, 0)
    yg = to_host(gpu.cnn_lrn_fwd(to_dev(x), size, alpha, beta, k))
    assert_elementwise_close(yg, oracle.lrn_fwd(x, size, alpha, beta, k), np.abs(x).max(), tag)
