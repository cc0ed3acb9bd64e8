"""C-ABI checks that need no GPU: the library loads, exports every function
include/cnn.h declares, its host-side shape helpers agree with the oracle's,
and invalid arguments are rejected before any launch.

No call here enqueues GPU work: every compute entry point is called only
with arguments that its host-side validation rejects.
"""
import ctypes
import os
import re

import pytest

import oracle
from paper_1511_07376_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cnn.h")

cnn = pytest.importorskip("paper_1511_07376_amd.cnn", reason="libcnn.so not built")

FAKE = 0x1000  # a non-null pointer that is never dereferenced (validation fails first)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*[A-Za-z_][\w\s\*]*?\b(cnn_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 13, names
    for name in names:
        assert hasattr(cnn.lib, name), f"{name} declared in cnn.h but not exported"
    assert set(names) == set(cnn.EXPORTED)


def test_version_and_empty_error():
    assert "gfx950" in cnn.cnn_version()


def test_layer_desc_layout_matches_header():
    # 13 int32 + 3 float + 2 int32 = 72 bytes, then three pointers
    assert ctypes.sizeof(cnn.cnn_layer_desc) == 96
    assert cnn.cnn_layer_desc.weight.offset == 72


@pytest.mark.parametrize("H,R,s,p", [(227, 11, 4, 0), (27, 5, 1, 2), (13, 3, 1, 1), (28, 5, 1, 0),
                                     (224, 7, 2, 3), (56, 1, 1, 0), (9, 4, 3, 2), (5, 5, 1, 0)])
def test_conv_out_shape_agrees_with_oracle(H, R, s, p):
    assert cnn.cnn_conv2d_out_shape(H, H + 3, R, R, s, p) == \
        oracle.conv2d_out_shape(H, H + 3, R, R, s, s, p, p)


def test_shape_arithmetic_near_int_max():
    """Extents near INT32_MAX are computed without wrapping: an output that
    does not fit is rejected, one that does is exact."""
    big = 2**31 - 1
    with pytest.raises(cnn.CnnError):
        cnn.cnn_conv2d_out_shape(1, 1, 1, 1, 1, big)          # 1 + 2*pad output rows
    assert cnn.cnn_conv2d_out_shape(big, 1, big, 1, 1, 0) == (1, 1)
    e = (big + 2 * 2**30 - 3) // 2**30 + 1                    # exact, 64-bit
    assert cnn.cnn_conv2d_out_shape(big, big, 3, 3, 2**30, 2**30) == (e, e)
    with pytest.raises(cnn.CnnError):
        cnn.cnn_pool_out_shape(big, 1, (2, 1), 1, (1, 0))      # 2^31 windows
    assert cnn.cnn_pool_out_shape(big, big, big, big, 0, True) == (1, 1)


def test_pool_out_shape_agrees_with_oracle_exhaustive():
    for H in range(1, 20):
        for k in range(1, 5):
            for s in range(1, 5):
                for p in range(0, k):
                    for ceil in (True, False):
                        if H + 2 * p < k:
                            continue
                        assert cnn.cnn_pool_out_shape(H, H, k, s, p, ceil) == \
                            oracle.pool_out_shape(H, H, k, k, s, s, p, p, ceil), (H, k, s, p, ceil)


@pytest.mark.parametrize("name,out", [("lenet", (16, 10)), ("cifar_quick", (32, 10)),
                                      ("alexnet", (64, 1000))])
def test_net_out_shape_and_workspace(name, out):
    net = wl.NETS[name]
    descs = _descs(net)
    C, H, W = net.input_chw
    oc, oh, ow = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    rc = cnn.lib.cnn_net_out_shape(descs, len(descs), out[0], C, H, W, ctypes.byref(oc),
                                   ctypes.byref(oh), ctypes.byref(ow))
    assert rc == 0, cnn.cnn_last_error()
    assert (oc.value, oh.value, ow.value) == (out[1], 1, 1)
    ws = cnn.lib.cnn_net_workspace_bytes(descs, len(descs), out[0], C, H, W)
    # two 256-byte aligned buffers of the largest activation, then one aligned
    # output per FC layer other than the last (at these batches every FC layer
    # splits its reduction: its output tiles cannot fill the GPU), and one per
    # conv layer that some tile configuration would split
    outs = oracle.net_fwd(net, wl.make_input(net, 1), wl.make_params(net), keep=True)[1]
    half = (max(a.size for a in outs) * out[0] * 4 + 255) // 256 * 256
    al = lambda b: (b + 255) // 256 * 256
    fc_area = sum(al(out[0] * l.out_features * 4) for l in [l for l in net.layers if l.kind == "fc"][:-1])
    conv_outs = [al(a.size * out[0] * 4) for l, a in zip(net.layers, outs) if l.kind == "conv"]
    sums = {0}
    for b in conv_outs:
        sums |= {s + b for s in sums}
    assert ws - 2 * half - fc_area in sums


def _descs(net):
    """Descriptors with fake (never dereferenced) weight pointers."""
    descs = (cnn.cnn_layer_desc * len(net.layers))()
    for i, layer in enumerate(net.layers):
        d = descs[i]
        if layer.kind == "conv":
            d.type, d.out_channels = cnn.CNN_LAYER_CONV, layer.out_channels
            d.in_channels = layer.in_channels
            d.kernel_h, d.kernel_w = layer.kernel
            d.stride_h, d.stride_w = layer.stride
            d.pad_h, d.pad_w = layer.pad
            d.groups, d.fuse_relu, d.weight = layer.groups, int(layer.relu), FAKE
        elif layer.kind == "fc":
            d.type, d.out_channels, d.in_features = cnn.CNN_LAYER_FC, layer.out_features, layer.in_features
            d.fuse_relu, d.weight = int(layer.relu), FAKE
        elif layer.kind == "pool":
            d.type = cnn.CNN_LAYER_POOL
            d.pool_mode = 0 if layer.mode == "max" else 1
            d.kernel_h, d.kernel_w = layer.kernel
            d.stride_h, d.stride_w = layer.stride
            d.pad_h, d.pad_w = layer.pad
            d.ceil_mode, d.fuse_relu = int(layer.ceil), int(layer.relu)
        elif layer.kind == "lrn":
            d.type, d.lrn_size = cnn.CNN_LAYER_LRN, layer.size
            d.lrn_alpha, d.lrn_beta, d.lrn_k = layer.alpha, layer.beta, layer.k
        elif layer.kind == "softmax":
            d.type = cnn.CNN_LAYER_SOFTMAX
        else:
            d.type = cnn.CNN_LAYER_RELU
    return descs


# ---------------------------------------------------------------- rejected arguments
L = cnn.lib


@pytest.mark.parametrize("args,status", [
    # (x, N, C, H, W, w, K, R, S, bias, sh, sw, ph, pw, G, relu, y, stream)
    ((0, 1, 3, 8, 8, FAKE, 4, 3, 3, 0, 1, 1, 0, 0, 1, 0, FAKE, 0), cnn.CNN_ERR_INVALID),       # null x
    ((FAKE, 1, 3, 8, 8, FAKE, 4, 3, 3, 0, 1, 1, 0, 0, 1, 0, 0, 0), cnn.CNN_ERR_INVALID),       # null y
    ((FAKE, 1, 3, 8, 8, FAKE, 4, 3, 3, 0, 0, 1, 0, 0, 1, 0, FAKE, 0), cnn.CNN_ERR_INVALID),    # stride 0
    ((FAKE, 1, 3, 8, 8, FAKE, 4, 3, 3, 0, 1, 1, 0, 0, 2, 0, FAKE, 0), cnn.CNN_ERR_INVALID),    # 2 !| 3
    ((FAKE, 1, 4, 8, 8, FAKE, 6, 3, 3, 0, 1, 1, 0, 0, 4, 0, FAKE, 0), cnn.CNN_ERR_INVALID),    # 4 !| 6
    ((FAKE, 1, 3, 2, 2, FAKE, 4, 3, 3, 0, 1, 1, 0, 0, 1, 0, FAKE, 0), cnn.CNN_ERR_INVALID),    # kernel > input
    ((FAKE, -1, 3, 8, 8, FAKE, 4, 3, 3, 0, 1, 1, 0, 0, 1, 0, FAKE, 0), cnn.CNN_ERR_INVALID),   # N < 0
    ((FAKE, 1, 3, 8, 8, FAKE, 4, 3, 3, 0, 1, 1, -1, 0, 1, 0, FAKE, 0), cnn.CNN_ERR_INVALID),   # pad < 0
    ((FAKE, 70000, 64, 224, 224, FAKE, 4, 3, 3, 0, 1, 1, 1, 1, 1, 0, FAKE, 0), cnn.CNN_ERR_UNSUPPORTED),
])
def test_conv_rejects(args, status):
    assert L.cnn_conv2d_fwd(*args) == status
    assert cnn.cnn_last_error().startswith("conv")


def test_fc_pool_lrn_relu_reject():
    assert L.cnn_fc_fwd(FAKE, 4, 0, FAKE, 0, 10, 0, FAKE, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_fc_fwd(0, 4, 8, FAKE, 0, 10, 0, FAKE, 0) == cnn.CNN_ERR_INVALID
    # pool: pad must be below the window; indices need max mode; bad mode
    assert L.cnn_pool_fwd(FAKE, 1, 1, 8, 8, 0, 2, 2, 2, 2, 2, 0, 1, 0, FAKE, 0, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_pool_fwd(FAKE, 1, 1, 8, 8, 1, 2, 2, 2, 2, 0, 0, 1, 0, FAKE, FAKE, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_pool_fwd(FAKE, 1, 1, 8, 8, 7, 2, 2, 2, 2, 0, 0, 1, 0, FAKE, 0, 0) == cnn.CNN_ERR_INVALID
    # input within 2^31-1 elements (46340^2), padded 2x2/1 output not (46341^2)
    assert L.cnn_pool_fwd(FAKE, 1, 1, 46340, 46340, 0, 2, 2, 1, 1, 1, 1, 1, 0, FAKE, 0, 0) == \
        cnn.CNN_ERR_UNSUPPORTED
    assert L.cnn_lrn_fwd(FAKE, 1, 4, 4, 4, 4, 1e-4, 0.75, 1.0, FAKE, 0) == cnn.CNN_ERR_UNSUPPORTED
    assert L.cnn_lrn_fwd(FAKE, 1, 4, 4, 4, 0, 1e-4, 0.75, 1.0, FAKE, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_relu_fwd(FAKE, FAKE, -1, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_relu_fwd(0, FAKE, 4, 0) == cnn.CNN_ERR_INVALID


def test_softmax_rejects():
    assert L.cnn_softmax_fwd(FAKE, -1, 10, 1, FAKE, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_softmax_fwd(FAKE, 2, 0, 1, FAKE, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_softmax_fwd(FAKE, 2, 10, 0, FAKE, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_softmax_fwd(0, 2, 10, 1, FAKE, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_softmax_fwd(FAKE, 70000, 1000, 100, FAKE, 0) == cnn.CNN_ERR_UNSUPPORTED
    # partial overlap (y four floats past x) is refused; N = 0 enqueues nothing
    assert L.cnn_softmax_fwd(FAKE, 2, 10, 1, FAKE + 16, 0) == cnn.CNN_ERR_INVALID
    assert "overlap" in cnn.cnn_last_error()
    assert L.cnn_softmax_fwd(0, 0, 10, 1, 0, 0) == cnn.CNN_OK


def test_net_with_softmax_layers_out_shape():
    """Softmax keeps the shape: after FC [N][O], after a conv [N][C][H][W]."""
    net = wl.Net("sm", (3, 12, 12), (wl.conv(3, 6, 3), wl.softmax(), wl.pool("max", 2, 2),
                                     wl.fc(6 * 5 * 5, 7), wl.softmax()), 0.1, 0.1)
    descs = _descs(net)
    oc, oh, ow = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    assert L.cnn_net_out_shape(descs, len(descs), 4, 3, 12, 12, ctypes.byref(oc), ctypes.byref(oh),
                               ctypes.byref(ow)) == 0, cnn.cnn_last_error()
    assert (oc.value, oh.value, ow.value) == (7, 1, 1)
    assert L.cnn_net_out_shape(descs, 2, 4, 3, 12, 12, ctypes.byref(oc), ctypes.byref(oh),
                               ctypes.byref(ow)) == 0
    assert (oc.value, oh.value, ow.value) == (6, 10, 10)


def test_net_rejects_before_launch():
    net = wl.alexnet
    C, H, W = net.input_chw
    descs = _descs(net)
    n = len(descs)
    # workspace too small
    assert L.cnn_net_fwd(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1024, 0) == cnn.CNN_ERR_WORKSPACE
    assert "workspace" in cnn.cnn_last_error()
    # FC input size inconsistent with the layer chain
    descs[10].in_features = 9000
    assert L.cnn_net_fwd(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, 0) == cnn.CNN_ERR_INVALID
    assert "layer 10" in cnn.cnn_last_error()
    descs[10].in_features = 9216
    # missing weights
    descs[0].weight = None
    assert L.cnn_net_fwd(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, 0) == cnn.CNN_ERR_INVALID
    descs[0].weight = FAKE
    # unknown layer type, no layers, input channels different from the first conv's
    descs[1].type = 9
    assert L.cnn_net_fwd(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, 0) == cnn.CNN_ERR_INVALID
    descs[1].type = cnn.CNN_LAYER_LRN
    assert L.cnn_net_fwd(descs, 0, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_net_fwd(descs, n, FAKE, 2, 4, H, W, FAKE, FAKE, 1 << 40, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_net_fwd_timed(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, None, 0) == cnn.CNN_ERR_INVALID
    # kernel-timestamp spans: both arrays, two distinct non-null events per layer
    evs = (ctypes.c_void_p * n)(*[FAKE + 16 * i for i in range(n)])
    evs2 = (ctypes.c_void_p * n)(*[FAKE + 16 * (n + i) for i in range(n)])
    assert L.cnn_net_fwd_kernel_timed(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, None, evs2, 0) == \
        cnn.CNN_ERR_INVALID
    assert L.cnn_net_fwd_kernel_timed(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, evs, None, 0) == \
        cnn.CNN_ERR_INVALID
    assert L.cnn_net_fwd_kernel_timed(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, evs, evs, 0) == \
        cnn.CNN_ERR_INVALID
    assert "two distinct events" in cnn.cnn_last_error()
    evs2[3] = None
    assert L.cnn_net_fwd_kernel_timed(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, evs, evs2, 0) == \
        cnn.CNN_ERR_INVALID
    assert "layer 3" in cnn.cnn_last_error()
    assert L.cnn_net_fwd_kernel_timed(descs, 5000, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, evs, evs2, 0) == \
        cnn.CNN_ERR_UNSUPPORTED
    assert L.cnn_net_fwd_dump(descs, n, FAKE, 2, C, H, W, FAKE, FAKE, 1 << 40, None, None, 0) == \
        cnn.CNN_ERR_INVALID
    assert "dump" in cnn.cnn_last_error()
    # the no-allocation pass: validated like cnn_net_fwd, and a workspace
    # beyond the static scratch is refused before any device call
    assert L.cnn_net_fwd_noalloc(descs, 0, FAKE, 2, C, H, W, FAKE, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_net_workspace_bytes(descs, n, 128, C, H, W) > cnn.CNN_NOALLOC_SCRATCH_BYTES
    assert L.cnn_net_fwd_noalloc(descs, n, FAKE, 128, C, H, W, FAKE, 0) == cnn.CNN_ERR_WORKSPACE
    assert "static scratch" in cnn.cnn_last_error()
    assert L.cnn_net_workspace_bytes(descs, 0, 2, C, H, W) == 0


def test_tuning_table_text_roundtrip():
    """Import / export / clear of the tuning records: host-only, no launches."""
    assert cnn.cnn_conv2d_num_configs() >= 4
    assert cnn.cnn_conv2d_config_name(0)
    assert cnn.cnn_conv2d_config_name(-5) is None
    cnn.cnn_tuning_clear()
    assert cnn.cnn_tuning_export() == ""
    n = cnn.cnn_tuning_import("# comment\n64 3 227 227 96 11 11 4 4 0 0 1 2\n64 256 13 13 384 3 3 1 1 1 1 1 0\n")
    assert n == 2
    text = cnn.cnn_tuning_export()
    assert "64 3 227 227 96 11 11 4 4 0 0 1 2\n" in text and text.count("\n") == 2
    with pytest.raises(cnn.CnnError):
        cnn.cnn_tuning_import("1 2 3\n")
    with pytest.raises(cnn.CnnError):
        cnn.cnn_tuning_import(f"1 3 8 8 4 3 3 1 1 0 0 1 {cnn.cnn_conv2d_num_configs()}\n")
    assert L.cnn_set_autotune(7) == cnn.CNN_ERR_INVALID
    assert L.cnn_conv2d_fwd_config(FAKE, 1, 3, 8, 8, FAKE, 4, 3, 3, 0, 1, 1, 0, 0, 1, 0, FAKE, 999, 0) \
        == cnn.CNN_ERR_INVALID
    cnn.cnn_tuning_clear()
    assert cnn.cnn_tuning_export() == ""


def test_fc_config_table_and_rejects():
    """FC configuration names and argument checks: host-only, no launches."""
    n = cnn.cnn_fc_num_configs()
    assert n >= 3 and all(cnn.cnn_fc_config_name(i) for i in range(n))
    assert cnn.cnn_fc_config_name(n) is None and cnn.cnn_fc_config_name(-1) is None
    assert L.cnn_fc_fwd_config(FAKE, 4, 8, FAKE, 0, 10, 0, FAKE, n, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_fc_fwd_config(FAKE, 4, 8, FAKE, 0, 10, 0, FAKE, -2, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_fc_fwd_config(FAKE, 4, 0, FAKE, 0, 10, 0, FAKE, 0, 0) == cnn.CNN_ERR_INVALID
    assert L.cnn_fc_fwd_config(0, 4, 8, FAKE, 0, 10, 0, FAKE, 0, 0) == cnn.CNN_ERR_INVALID


def test_workspace_holds_bordered_pool_output():
    """A padded conv after LRN + pooling reads the pooled planes inside their
    zero border: the workspace holds two buffers of the bordered size when
    that is the largest activation (8 x 34 x 34 here, against 8 x 30 x 30 for
    the LRN and the 3x3/1 pooling and 4 x 30 x 30 out of the conv, the last
    layer)."""
    net = wl.Net("lrn_pool_conv", (8, 30, 30), (
        wl.lrn(5, 1e-4, 0.75, 1.0), wl.pool("max", 3, 1, 1), wl.conv(8, 4, 5, 1, 2)), 0.1, 0.1)
    descs = _descs(net)
    for N in (1, 7, 64):
        ws = cnn.lib.cnn_net_workspace_bytes(descs, len(descs), N, 8, 30, 30)
        half = (N * 8 * 34 * 34 * 4 + 255) // 256 * 256
        assert ws == 2 * half, (N, ws, half)
    # without the LRN the pooling kernel writes plain planes (and the conv pads)
    plain = wl.Net("pool_conv", (8, 30, 30), (wl.pool("max", 3, 1, 1), wl.conv(8, 4, 5, 1, 2)), 0.1, 0.1)
    descs = _descs(plain)
    ws = cnn.lib.cnn_net_workspace_bytes(descs, len(descs), 7, 8, 30, 30)
    assert ws == 2 * ((7 * 8 * 30 * 30 * 4 + 255) // 256 * 256)


def test_binding_refuses_to_load_without_the_library(tmp_path):
    """A copy of the package without libcnn.so raises on import: there is no
    fallback path that could compute anything without the HIP library."""
    import shutil
    import subprocess
    import sys
    pkg = os.path.join(ROOT, "paper_1511_07376_amd")
    dst = tmp_path / "paper_1511_07376_amd"
    shutil.copytree(pkg, dst, ignore=shutil.ignore_patterns("libcnn.so", "_build", "__pycache__", "csrc"))
    code = "import paper_1511_07376_amd.cnn"
    r = subprocess.run([sys.executable, "-c", code], cwd=tmp_path, capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "libcnn.so is missing" in r.stderr


def test_bordered_planning_with_extreme_padding():
    """The bordered input extent (pooled plane + 2 x pad) is formed in 64
    bits: with a padding near 2^30 (and a stride that keeps the conv output
    small) the planner falls back to the padded conv instead of wrapping."""
    net = wl.Net("x", (8, 30, 30), (wl.lrn(5, 1e-4, 0.75, 1.0), wl.pool("max", 3, 2),
                                     wl.conv(8, 4, 3, 2**30, 2**30)), 0.1, 0.1)
    descs = _descs(net)
    assert cnn.cnn_conv2d_out_shape(15, 15, 3, 3, 2**30, 2**30) == (3, 3)
    ws = cnn.lib.cnn_net_workspace_bytes(descs, len(descs), 2, 8, 30, 30)
    assert ws == 2 * ((2 * 8 * 30 * 30 * 4 + 255) // 256 * 256)  # the LRN's output is the largest
