"""Layers at the library's size limits (GPU): tensors of close to 2^31-1
elements, the most any single tensor may hold.

Each case is chosen so that a 32-bit index or loop counter would wrap:
- grid-stride loops whose last step passes 2^31: direct max/avg pooling
  (planes too large to stage), LRN of images of 2^29 or more elements;
- staged pooling of more than 2^30 planes;
- a convolution whose images are each just under 2^29 elements, so it runs
  as one launch per image;
- an FC layer whose input spans more than 2^31 bytes;
- a ReLU over more than 2^31 elements, aligned and not.

Inputs are generated on the device with a seeded torch generator (numpy at
these sizes would take minutes); the oracle gets copies of the same bytes.
Outputs start as NaN, so an element no thread wrote fails the full-size
property checks (every element: a window maximum is at least its centre, an
average of values in [0, 1) lies in [0, 1), ...).  Sampled planes, rows or
runs, first and last included, go through the oracle with the tolerances of
the other layer tests: max pooling values and indices bit-exact, average
pooling and LRN elementwise, conv and FC by the GEMM criterion.
"""
import gc

import numpy as np
import pytest

import oracle
from parity import assert_elementwise_close, assert_gemm_close

pytestmark = pytest.mark.gpu

INT_MAX = 2**31 - 1


def _torch():
    import torch
    return torch


def _rand(shape, seed, normal=False):
    torch = _torch()
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    if normal:
        return torch.randn(shape, generator=g, device="cuda")
    return torch.rand(shape, generator=g, device="cuda")


def _nan(shape):
    torch = _torch()
    return torch.full(shape, float("nan"), device="cuda")


def _host(t):
    torch = _torch()
    torch.cuda.synchronize()
    return t.cpu().numpy()


@pytest.fixture(autouse=True)
def _release():
    yield
    gc.collect()
    _torch().cuda.empty_cache()


def test_pool_direct_near_int_max(gpu):
    """3x3/1 pad 1 pooling of 2,015,821,824 elements in 128x128 planes (too
    large to stage in LDS): one thread per output in a grid-stride loop whose
    last step passes 2^31."""
    torch = _torch()
    N, C, H, W = 31, 3969, 128, 128
    total = N * C * H * W
    assert INT_MAX - 2**28 < total <= INT_MAX
    print(f"pool direct {N}x{C}x{H}x{W} max", flush=True)
    x = _rand((N, C, H, W), 21)
    y = _nan((N, C, H, W))
    idx = torch.full((N, C, H, W), -1, dtype=torch.int32, device="cuda")
    gpu.cnn_pool_fwd(x, "max", 3, 1, 1, True, with_index=True, y=y, idx=idx)
    torch.cuda.synchronize()
    assert bool((y >= x).all()), "an output below its window's centre (or never written)"
    assert bool(((idx >= 0) & (idx < H * W)).all())
    xf, yf, jf = x.view(N * C, H * W), y.view(N * C, H * W), idx.view(N * C, H * W)
    for c0 in range(0, N * C, 16384):  # y == x[idx], in slices of planes
        c1 = min(c0 + 16384, N * C)
        assert torch.equal(xf[c0:c1].gather(1, jf[c0:c1].long()), yf[c0:c1]), c0
    for n, c in ((0, 0), (15, 2000), (N - 1, C - 1)):
        xs = _host(x[n:n + 1, c:c + 1])
        ry, ri = oracle.pool_fwd(xs, "max", (3, 3), (1, 1), (1, 1), True, with_index=True)
        np.testing.assert_array_equal(_host(y[n:n + 1, c:c + 1]), ry)
        np.testing.assert_array_equal(_host(idx[n:n + 1, c:c + 1]), ri)
    del idx
    print(f"pool direct {N}x{C}x{H}x{W} avg", flush=True)
    y.fill_(float("nan"))
    gpu.cnn_pool_fwd(x, "avg", 3, 1, 1, True, y=y)
    torch.cuda.synchronize()
    assert bool(((y >= 0) & (y < 1)).all()), "an average outside [0, 1) (or never written)"
    for n, c in ((0, 0), (15, 2000), (N - 1, C - 1)):
        xs = _host(x[n:n + 1, c:c + 1])
        ry = oracle.pool_fwd(xs, "avg", (3, 3), (1, 1), (1, 1), True)
        assert_elementwise_close(_host(y[n:n + 1, c:c + 1]), ry, 1.0, f"avg plane {n},{c}")


def test_pool_staged_over_2pow30_planes(gpu):
    """2,000,000,000 planes of one element, staged 4096 planes per workgroup:
    the loop over plane runs steps past 2^31.  A 1x1 window is the identity
    (index 0), for max and average alike."""
    torch = _torch()
    C = 2_000_000_000
    print(f"pool staged 1x{C}x1x1", flush=True)
    x = _rand((1, C, 1, 1), 22)
    y = _nan((1, C, 1, 1))
    idx = torch.full((1, C, 1, 1), -1, dtype=torch.int32, device="cuda")
    gpu.cnn_pool_fwd(x, "max", 1, 1, 0, True, with_index=True, y=y, idx=idx)
    torch.cuda.synchronize()
    assert torch.equal(y, x)
    assert bool((idx == 0).all())
    for sl in (slice(0, 4096), slice(C - 4096, C)):
        ry, ri = oracle.pool_fwd(_host(x[:, sl]), "max", (1, 1), (1, 1), (0, 0), True, with_index=True)
        np.testing.assert_array_equal(_host(y[:, sl]), ry)
        np.testing.assert_array_equal(_host(idx[:, sl]), ri)
    del idx
    y.fill_(float("nan"))
    gpu.cnn_pool_fwd(x, "avg", 1, 1, 0, True, y=y)
    torch.cuda.synchronize()
    assert torch.equal(y, x)


def test_lrn_huge_image(gpu):
    """LRN of one 45000x45000 image (2,025,000,000 elements, 2^29 or more per
    image: the unchunked kernel), one channel, so each output is the closed
    form x (k + alpha/n x^2)^-beta."""
    torch = _torch()
    shape = (1, 1, 45000, 45000)
    print(f"lrn {shape}", flush=True)
    x = _rand(shape, 23)
    y = _nan(shape)
    gpu.cnn_lrn_fwd(x, 5, 1e-2, 0.75, 2.0, y=y)
    torch.cuda.synchronize()
    assert bool(((y >= 0) & (y <= x)).all()), "k = 2 shrinks every value (or it was never written)"
    flat_x, flat_y = x.view(-1), y.view(-1)
    n = flat_x.numel()
    for a in (0, n // 2, n - 4096):
        xs = _host(flat_x[a:a + 4096]).reshape(1, 1, 1, 4096)
        ref = oracle.lrn_fwd(xs, 5, 1e-2, 0.75, 2.0)
        assert_elementwise_close(_host(flat_y[a:a + 4096]).reshape(ref.shape), ref, 1.0, f"lrn run {a}")


def test_conv_one_launch_per_image(gpu):
    """3x3/2 pad 1 convolution of 4 images of 8x8191x8192 (536,805,376
    elements each, just under 2^29): one launch per image, 8.6 GB of input."""
    torch = _torch()
    N, C, H, W, K = 4, 8, 8191, 8192, 4
    print(f"conv {N}x{C}x{H}x{W} K{K} 3x3/2 p1", flush=True)
    x = _rand((N, C, H, W), 24, normal=True)
    wgt = _rand((K, C, 3, 3), 25, normal=True)
    b = _rand((K,), 26, normal=True)
    P, Q = gpu.cnn_conv2d_out_shape(H, W, 3, 3, 2, 1)
    assert (P, Q) == (4096, 4096)
    y = _nan((N, K, P, Q))
    gpu.cnn_conv2d_fwd(x, wgt, b, stride=2, pad=1, y=y)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all()), "an output never written"
    wh, bh = _host(wgt), _host(b)
    for n in (0, N - 1):
        for p in (0, 2047, P - 1):
            rows = np.zeros((1, C, 3, W), np.float32)  # input rows 2p-1 .. 2p+1, zero outside
            for r in range(3):
                h = 2 * p - 1 + r
                if 0 <= h < H:
                    rows[0, :, r] = _host(x[n, :, h])
            ref = oracle.conv2d_fwd(rows, wh, bh, stride=(2, 2), pad=(0, 1))
            assert_gemm_close(_host(y[n:n + 1, :, p:p + 1]), ref, C * 9, f"conv n{n} row {p}")


def test_fc_input_beyond_2pow31_bytes(gpu):
    """FC of 262,143 images of 8192 features (2,147,475,456 elements: 8.6 GB,
    a ragged last tile of 63 images) to 64 outputs."""
    torch = _torch()
    N, I, O = 262143, 8192, 64
    assert N * I <= INT_MAX
    print(f"fc {N}x{I} -> {O}", flush=True)
    x = _rand((N, I), 27, normal=True)
    wgt = _rand((O, I), 28, normal=True) * 0.01
    b = _rand((O,), 29, normal=True)
    y = _nan((N, O))
    gpu.cnn_fc_fwd(x, wgt, b, fuse_relu=True, y=y)
    torch.cuda.synchronize()
    assert bool((y >= 0).all()), "a negative or NaN output (ReLU fused; never written)"
    wh, bh = _host(wgt), _host(b)
    for rows in (slice(0, 64), slice(N // 2, N // 2 + 64), slice(N - 64, N)):
        ref = oracle.fc_fwd(_host(x[rows]), wh, bh, relu=True)
        assert_gemm_close(_host(y[rows]), ref, I, f"fc rows {rows.start}")


@pytest.mark.parametrize("offset", [0, 1])
def test_relu_beyond_int32(gpu, offset):
    """ReLU over 2^31 + 5 elements: a 16-byte aligned run (vector kernel, then
    a tail of 1) and, from one element in, an unaligned one; in place for the
    second."""
    torch = _torch()
    n = 2**31 + 5
    print(f"relu n={n} offset {offset}", flush=True)
    base = _rand((n + offset,), 30, normal=True)
    x = base[offset:]
    if offset:
        keep = _host(x[-4096:]).copy()
        head = _host(x[:4096]).copy()
        gpu.cnn_relu_fwd(x, y=x)
        torch.cuda.synchronize()
        assert bool((x >= 0).all())
        np.testing.assert_array_equal(_host(x[-4096:]), oracle.relu_fwd(keep))
        np.testing.assert_array_equal(_host(x[:4096]), oracle.relu_fwd(head))
    else:
        y = _nan((n,))
        gpu.cnn_relu_fwd(x, y=y)
        torch.cuda.synchronize()
        assert torch.equal(y, x.clamp_min(0))
        np.testing.assert_array_equal(_host(y[-4096:]), oracle.relu_fwd(_host(x[-4096:])))
