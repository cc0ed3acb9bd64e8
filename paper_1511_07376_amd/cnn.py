"""Python binding of libcnn (include/cnn.h): argument marshalling only.

Every function here checks that its tensors are contiguous float32 CUDA
(ROCm) tensors, passes their device pointers and the current torch stream to
the C entry point of the same name, and raises ``CnnError`` with
``cnn_last_error()`` on a non-OK status.  All computation happens in the HIP
kernels of libcnn; torch provides device memory and the stream.  Importing
this module fails if libcnn.so has not been built.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import torch

from . import workloads as _wl

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcnn.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python __graft_entry__.py` "
                      "(or paper_1511_07376_amd/build.py) before using the GPU path")

lib = ctypes.CDLL(LIB_PATH)

_i = ctypes.c_int
_p = ctypes.c_void_p
_ip = ctypes.POINTER(ctypes.c_int)

CNN_OK, CNN_ERR_INVALID, CNN_ERR_UNSUPPORTED, CNN_ERR_HIP, CNN_ERR_WORKSPACE = 0, -1, -2, -3, -4
CNN_POOL_MAX, CNN_POOL_AVG = 0, 1
CNN_LAYER_CONV, CNN_LAYER_FC, CNN_LAYER_POOL, CNN_LAYER_LRN, CNN_LAYER_RELU = 0, 1, 2, 3, 4
CNN_LAYER_SOFTMAX = 5


class cnn_layer_desc(ctypes.Structure):
    _fields_ = [
        ("type", ctypes.c_int32), ("out_channels", ctypes.c_int32),
        ("kernel_h", ctypes.c_int32), ("kernel_w", ctypes.c_int32),
        ("stride_h", ctypes.c_int32), ("stride_w", ctypes.c_int32),
        ("pad_h", ctypes.c_int32), ("pad_w", ctypes.c_int32),
        ("groups", ctypes.c_int32), ("pool_mode", ctypes.c_int32),
        ("ceil_mode", ctypes.c_int32), ("fuse_relu", ctypes.c_int32),
        ("lrn_size", ctypes.c_int32), ("lrn_alpha", ctypes.c_float),
        ("lrn_beta", ctypes.c_float), ("lrn_k", ctypes.c_float),
        ("in_channels", ctypes.c_int32), ("in_features", ctypes.c_int32),
        ("weight", ctypes.c_void_p), ("bias", ctypes.c_void_p), ("pool_index", ctypes.c_void_p),
    ]


lib.cnn_conv2d_out_shape.argtypes = [_i] * 8 + [_ip, _ip]
lib.cnn_pool_out_shape.argtypes = [_i] * 9 + [_ip, _ip]
lib.cnn_conv2d_fwd.argtypes = [_p, _i, _i, _i, _i, _p, _i, _i, _i, _p, _i, _i, _i, _i, _i, _i, _p, _p]
lib.cnn_fc_fwd.argtypes = [_p, _i, _i, _p, _p, _i, _i, _p, _p]
lib.cnn_pool_fwd.argtypes = [_p, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _p, _p, _p]
lib.cnn_lrn_fwd.argtypes = [_p, _i, _i, _i, _i, _i, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                            _p, _p]
lib.cnn_relu_fwd.argtypes = [_p, _p, ctypes.c_int64, _p]
lib.cnn_softmax_fwd.argtypes = [_p, _i, _i, _i, _p, _p]


class cnn_netfile_config(ctypes.Structure):
    _fields_ = [("in_channels", ctypes.c_int32), ("in_height", ctypes.c_int32),
                ("in_width", ctypes.c_int32), ("execution_mode", ctypes.c_int32),
                ("auto_tuning", ctypes.c_int32), ("allocated_ram_mib", ctypes.c_int32)]


CNN_EXEC_PARALLEL, CNN_EXEC_GRAPH = 0, 1
_descp = ctypes.POINTER(cnn_layer_desc)
lib.cnn_net_out_shape.argtypes = [_descp, _i, _i, _i, _i, _i, _ip, _ip, _ip]
lib.cnn_net_workspace_bytes.argtypes = [_descp, _i, _i, _i, _i, _i]
lib.cnn_net_workspace_bytes.restype = ctypes.c_size_t
lib.cnn_net_fwd.argtypes = [_descp, _i, _p, _i, _i, _i, _i, _p, _p, ctypes.c_size_t, _p]
lib.cnn_net_fwd_timed.argtypes = [_descp, _i, _p, _i, _i, _i, _i, _p, _p, ctypes.c_size_t,
                                  ctypes.POINTER(ctypes.c_void_p), _p]
lib.cnn_net_fwd_kernel_timed.argtypes = [_descp, _i, _p, _i, _i, _i, _i, _p, _p, ctypes.c_size_t,
                                         ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(ctypes.c_void_p), _p]
lib.cnn_net_fwd_dump.argtypes = [_descp, _i, _p, _i, _i, _i, _i, _p, _p, ctypes.c_size_t,
                                 ctypes.POINTER(ctypes.c_void_p), _ip, _p]
lib.cnn_net_fwd_noalloc.argtypes = [_descp, _i, _p, _i, _i, _i, _i, _p, _p]
CNN_NOALLOC_SCRATCH_BYTES = 256 << 20
lib.cnn_conv2d_fwd_config.argtypes = lib.cnn_conv2d_fwd.argtypes[:17] + [_i, _p]
lib.cnn_netfile_parse.argtypes = [ctypes.c_char_p, _descp, _i, _ip, ctypes.POINTER(cnn_netfile_config)]
lib.cnn_net_graph_create.argtypes = [_descp, _i, _p, _i, _i, _i, _i, _p, _p, ctypes.c_size_t,
                                     ctypes.POINTER(ctypes.c_void_p)]
lib.cnn_net_graph_launch.argtypes = [_p, _p]
lib.cnn_net_graph_destroy.argtypes = [_p]
lib.cnn_conv2d_num_configs.argtypes = []
lib.cnn_conv2d_config_name.argtypes = [_i]
lib.cnn_conv2d_config_name.restype = ctypes.c_char_p
lib.cnn_fc_fwd_config.argtypes = lib.cnn_fc_fwd.argtypes[:8] + [_i, _p]
lib.cnn_fc_num_configs.argtypes = []
lib.cnn_fc_config_name.argtypes = [_i]
lib.cnn_fc_config_name.restype = ctypes.c_char_p
lib.cnn_set_autotune.argtypes = [_i]
lib.cnn_tuning_export.argtypes = [ctypes.c_char_p, ctypes.c_size_t]
lib.cnn_tuning_export.restype = ctypes.c_size_t
lib.cnn_tuning_import.argtypes = [ctypes.c_char_p]
lib.cnn_tuning_clear.argtypes = []
lib.cnn_last_error.restype = ctypes.c_char_p
lib.cnn_version.restype = ctypes.c_char_p
for _name in ("cnn_conv2d_out_shape", "cnn_pool_out_shape", "cnn_conv2d_fwd", "cnn_fc_fwd",
              "cnn_pool_fwd", "cnn_lrn_fwd", "cnn_relu_fwd", "cnn_softmax_fwd", "cnn_net_out_shape",
              "cnn_net_fwd",
              "cnn_net_fwd_timed", "cnn_net_fwd_kernel_timed", "cnn_net_fwd_dump", "cnn_net_fwd_noalloc",
              "cnn_conv2d_fwd_config",
              "cnn_conv2d_num_configs", "cnn_fc_fwd_config", "cnn_fc_num_configs",
              "cnn_set_autotune", "cnn_tuning_import", "cnn_tuning_clear", "cnn_netfile_parse",
              "cnn_net_graph_create", "cnn_net_graph_launch", "cnn_net_graph_destroy"):
    getattr(lib, _name).restype = _i

EXPORTED = ("cnn_conv2d_out_shape", "cnn_pool_out_shape", "cnn_conv2d_fwd", "cnn_fc_fwd",
            "cnn_pool_fwd", "cnn_lrn_fwd", "cnn_relu_fwd", "cnn_softmax_fwd", "cnn_net_out_shape",
            "cnn_net_workspace_bytes", "cnn_net_fwd", "cnn_net_fwd_timed", "cnn_net_fwd_kernel_timed",
            "cnn_net_fwd_dump",
            "cnn_net_fwd_noalloc", "cnn_last_error",
            "cnn_version", "cnn_conv2d_num_configs", "cnn_conv2d_config_name",
            "cnn_conv2d_fwd_config", "cnn_fc_num_configs", "cnn_fc_config_name", "cnn_fc_fwd_config",
            "cnn_set_autotune", "cnn_tuning_export",
            "cnn_tuning_import", "cnn_tuning_clear", "cnn_netfile_parse", "cnn_net_graph_create",
            "cnn_net_graph_launch", "cnn_net_graph_destroy")


class CnnError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libcnn status {status}: {message}")
        self.status = status


def cnn_last_error() -> str:
    # the message may quote the caller's text (a NetFile line), which need not be UTF-8
    return lib.cnn_last_error().decode(errors="replace")


def cnn_version() -> str:
    return lib.cnn_version().decode()


def _ok(rc: int) -> None:
    if rc != CNN_OK:
        raise CnnError(rc, cnn_last_error())


def _dev(t: Optional[torch.Tensor], name: str, dtype=torch.float32):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise TypeError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _pair(v) -> Tuple[int, int]:
    return (int(v), int(v)) if isinstance(v, int) else (int(v[0]), int(v[1]))


def cnn_conv2d_out_shape(H, W, R, S, stride=1, pad=0) -> Tuple[int, int]:
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    P, Q = ctypes.c_int(), ctypes.c_int()
    _ok(lib.cnn_conv2d_out_shape(H, W, R, S, sh, sw, ph, pw, ctypes.byref(P), ctypes.byref(Q)))
    return P.value, Q.value


def cnn_pool_out_shape(H, W, kernel, stride, pad=0, ceil_mode=True) -> Tuple[int, int]:
    kh, kw = _pair(kernel)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    P, Q = ctypes.c_int(), ctypes.c_int()
    _ok(lib.cnn_pool_out_shape(H, W, kh, kw, sh, sw, ph, pw, int(ceil_mode), ctypes.byref(P),
                               ctypes.byref(Q)))
    return P.value, Q.value


def cnn_conv2d_fwd(x, w, bias=None, stride=1, pad=0, groups=1, fuse_relu=False, y=None, stream=None,
                   config=None):
    """x [N][C][H][W], w [K][C/G][R][S], bias [K] -> y [N][K][P][Q] (allocated if None).

    config=None uses the tuned / heuristic tile configuration (cnn_conv2d_fwd);
    an int calls cnn_conv2d_fwd_config with that configuration (-1: heuristic)."""
    N, C, H, W = x.shape
    K, _cg, R, S = w.shape
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    if y is None:
        P, Q = cnn_conv2d_out_shape(H, W, R, S, (sh, sw), (ph, pw))
        y = torch.empty((N, K, P, Q), dtype=torch.float32, device=x.device)
    args = (_dev(x, "x"), N, C, H, W, _dev(w, "w"), K, R, S, _dev(bias, "bias"),
            sh, sw, ph, pw, groups, int(fuse_relu), _dev(y, "y"))
    if config is None:
        _ok(lib.cnn_conv2d_fwd(*args, _stream(stream)))
    else:
        _ok(lib.cnn_conv2d_fwd_config(*args, int(config), _stream(stream)))
    return y


def cnn_conv2d_num_configs() -> int:
    return int(lib.cnn_conv2d_num_configs())


def cnn_conv2d_config_name(i: int) -> Optional[str]:
    r = lib.cnn_conv2d_config_name(int(i))
    return None if r is None else r.decode()


def cnn_set_autotune(on: bool) -> None:
    _ok(lib.cnn_set_autotune(int(bool(on))))


def cnn_tuning_export() -> str:
    n = lib.cnn_tuning_export(None, 0)
    buf = ctypes.create_string_buffer(n)
    lib.cnn_tuning_export(buf, n)
    return buf.value.decode()


def cnn_tuning_import(text: str) -> int:
    rc = lib.cnn_tuning_import(text.encode())
    if rc < 0:
        raise CnnError(rc, cnn_last_error())
    return rc


def cnn_tuning_clear() -> None:
    _ok(lib.cnn_tuning_clear())


def cnn_fc_fwd(x, w, bias=None, fuse_relu=False, y=None, stream=None, config=None):
    """x [N][I] (or [N][C][H][W], read flattened), w [O][I] -> y [N][O].

    config=None calls cnn_fc_fwd (the built-in kernel choice); an int calls
    cnn_fc_fwd_config with that configuration (-1: the built-in choice)."""
    N = x.shape[0]
    I = x.numel() // max(N, 1) if N else int(w.shape[1])
    O = w.shape[0]
    if y is None:
        y = torch.empty((N, O), dtype=torch.float32, device=x.device)
    args = (_dev(x, "x"), N, I, _dev(w, "w"), _dev(bias, "bias"), O, int(fuse_relu), _dev(y, "y"))
    if config is None:
        _ok(lib.cnn_fc_fwd(*args, _stream(stream)))
    else:
        _ok(lib.cnn_fc_fwd_config(*args, int(config), _stream(stream)))
    return y


def cnn_fc_num_configs() -> int:
    return int(lib.cnn_fc_num_configs())


def cnn_fc_config_name(i: int) -> Optional[str]:
    r = lib.cnn_fc_config_name(int(i))
    return None if r is None else r.decode()


def cnn_pool_fwd(x, mode="max", kernel=2, stride=2, pad=0, ceil_mode=True, fuse_relu=False,
                 with_index=False, y=None, idx=None, stream=None):
    """Returns y, or (y, idx) for max pooling with with_index."""
    N, C, H, W = x.shape
    kh, kw = _pair(kernel)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    m = {"max": CNN_POOL_MAX, "avg": CNN_POOL_AVG}[mode] if isinstance(mode, str) else int(mode)
    P, Q = cnn_pool_out_shape(H, W, (kh, kw), (sh, sw), (ph, pw), ceil_mode)
    if y is None:
        y = torch.empty((N, C, P, Q), dtype=torch.float32, device=x.device)
    if with_index and idx is None:
        idx = torch.empty((N, C, P, Q), dtype=torch.int32, device=x.device)
    _ok(lib.cnn_pool_fwd(_dev(x, "x"), N, C, H, W, m, kh, kw, sh, sw, ph, pw, int(ceil_mode),
                         int(fuse_relu), _dev(y, "y"), _dev(idx, "idx", torch.int32), _stream(stream)))
    return (y, idx) if idx is not None else y


def cnn_lrn_fwd(x, size=5, alpha=1e-4, beta=0.75, k=1.0, y=None, stream=None):
    N, C, H, W = x.shape
    if y is None:
        y = torch.empty_like(x)
    _ok(lib.cnn_lrn_fwd(_dev(x, "x"), N, C, H, W, size, alpha, beta, k, _dev(y, "y"), _stream(stream)))
    return y


def cnn_relu_fwd(x, y=None, stream=None):
    """y = max(x, 0); pass y=x for in place."""
    if y is None:
        y = torch.empty_like(x)
    if y.numel() != x.numel():
        raise ValueError("relu: x and y differ in size")
    _ok(lib.cnn_relu_fwd(_dev(x, "x"), _dev(y, "y"), x.numel(), _stream(stream)))
    return y


def cnn_softmax_fwd(x, y=None, stream=None):
    """Softmax across dim 1 of an [N][C] or [N][C][H][W] tensor; pass y=x for
    in place."""
    if x.dim() < 2:
        raise ValueError("softmax: x must be [N][C...]")
    if y is None:
        y = torch.empty_like(x)
    if y.numel() != x.numel():
        raise ValueError("softmax: x and y differ in size")
    N, C = x.shape[0], x.shape[1]
    HW = 1
    for d in x.shape[2:]:
        HW *= d
    _ok(lib.cnn_softmax_fwd(_dev(x, "x"), N, C, HW, _dev(y, "y"), _stream(stream)))
    return y


# ---------------------------------------------------------------- NetFile
@dataclass(frozen=True)
class NetFile:
    """A parsed NetFile (cnn_netfile_parse): engine parameters and the layer
    list, as a ``workloads.Net`` whose layers carry the shapes that the
    library's own shape rules give for the declared input."""

    net: "_wl.Net"
    execution_mode: str
    auto_tuning: bool
    allocated_ram_mib: int


def parse_netfile(text: str, name: str = "netfile", input_chw: Optional[Tuple[int, int, int]] = None,
                  weight_std: float = 0.01, bias_std: float = 0.01) -> NetFile:
    """Parses NetFile text.  input_chw overrides (or supplies) the "input"
    statement; weight_std / bias_std only describe synthetic parameters."""
    raw = text.encode()
    n = ctypes.c_int()
    cfg = cnn_netfile_config()
    _ok(lib.cnn_netfile_parse(raw, None, 0, ctypes.byref(n), ctypes.byref(cfg)))
    descs = (cnn_layer_desc * max(n.value, 1))()
    _ok(lib.cnn_netfile_parse(raw, descs, n.value, ctypes.byref(n), ctypes.byref(cfg)))
    chw = input_chw or (cfg.in_channels, cfg.in_height, cfg.in_width)
    if min(chw) <= 0:
        raise ValueError("NetFile: no input shape (an 'input C H W' line or input_chw=)")
    layers = []
    shape = tuple(chw)
    oc, oh, ow = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    for i in range(n.value):
        d = descs[i]
        c, h, w = shape
        if d.type == CNN_LAYER_CONV:
            layers.append(_wl.conv(c, d.out_channels, (d.kernel_h, d.kernel_w), (d.stride_h, d.stride_w),
                                   (d.pad_h, d.pad_w), d.groups, bool(d.fuse_relu)))
        elif d.type == CNN_LAYER_FC:
            layers.append(_wl.fc(c * h * w, d.out_channels, bool(d.fuse_relu)))
        elif d.type == CNN_LAYER_POOL:
            layers.append(_wl.pool("max" if d.pool_mode == CNN_POOL_MAX else "avg", (d.kernel_h, d.kernel_w),
                                   (d.stride_h, d.stride_w), (d.pad_h, d.pad_w), bool(d.ceil_mode),
                                   bool(d.fuse_relu)))
        elif d.type == CNN_LAYER_LRN:
            layers.append(_wl.lrn(d.lrn_size, d.lrn_alpha, d.lrn_beta, d.lrn_k))
        elif d.type == CNN_LAYER_RELU:
            layers.append(_wl.relu())
        else:
            layers.append(_wl.softmax())
        # shape after this layer, by the library's rules (also checks in=)
        _ok(lib.cnn_net_out_shape(descs, i + 1, 1, *chw, ctypes.byref(oc), ctypes.byref(oh),
                                  ctypes.byref(ow)))
        shape = (oc.value, oh.value, ow.value)
    net = _wl.Net(name, tuple(chw), tuple(layers), weight_std, bias_std)
    mode = "graph" if cfg.execution_mode == CNN_EXEC_GRAPH else "parallel"
    return NetFile(net, mode, bool(cfg.auto_tuning), cfg.allocated_ram_mib)


def load_netfile(path: str, **kw) -> NetFile:
    with open(path) as f:
        return parse_netfile(f.read(), name=os.path.splitext(os.path.basename(path))[0], **kw)


NETFILE_DIR = os.path.join(HERE, "netfiles")


# ---------------------------------------------------------------- networks
class Network:
    """A layer-descriptor array bound to device-resident parameters.

    Built from a ``workloads.Net`` and its (weight, bias) list; parameters are
    copied to the device once (loading is outside the timed path, as in the
    paper's measurements).  ``pool_index=True`` allocates an int32 index
    output for every max-pooling layer (per batch size, on first use).

    execution_mode (the NetFile parameter): "parallel" enqueues the layers on
    every call (cnn_net_fwd); "graph" runs the first call for a given
    (input, output, batch) eagerly, captures it into a HIP graph
    (cnn_net_graph_create) and replays the graph from then on.  In graph mode
    an output allocated by the call (y=None) is a buffer reused by later
    calls of the same batch size.
    """

    def __init__(self, net, params, device="cuda", pool_index: bool = False,
                 execution_mode: str = "parallel"):
        if execution_mode not in ("parallel", "graph"):
            raise ValueError(f"execution_mode {execution_mode!r}: parallel or graph")
        self.execution_mode = execution_mode
        self._graphs: Dict[tuple, ctypes.c_void_p] = {}
        self._outs: Dict[int, torch.Tensor] = {}
        self.net = net
        self.device = torch.device(device)
        self.weights: List[Tuple[Optional[torch.Tensor], Optional[torch.Tensor]]] = []
        for layer, pr in zip(net.layers, params):
            if layer.has_params:
                self.weights.append((torch.from_numpy(pr[0]).to(self.device).contiguous(),
                                     torch.from_numpy(pr[1]).to(self.device).contiguous()))
            else:
                self.weights.append((None, None))
        self.pool_index = pool_index
        self.indices: List[Optional[torch.Tensor]] = [None] * len(net.layers)
        self.descs = (cnn_layer_desc * len(net.layers))()
        for i, (layer, (w, b)) in enumerate(zip(net.layers, self.weights)):
            d = self.descs[i]
            if layer.kind == "conv":
                d.type = CNN_LAYER_CONV
                d.in_channels = layer.in_channels
                d.out_channels = layer.out_channels
                d.kernel_h, d.kernel_w = layer.kernel
                d.stride_h, d.stride_w = layer.stride
                d.pad_h, d.pad_w = layer.pad
                d.groups = layer.groups
                d.fuse_relu = int(layer.relu)
            elif layer.kind == "fc":
                d.type = CNN_LAYER_FC
                d.out_channels = layer.out_features
                d.in_features = layer.in_features
                d.fuse_relu = int(layer.relu)
            elif layer.kind == "pool":
                d.type = CNN_LAYER_POOL
                d.pool_mode = CNN_POOL_MAX if layer.mode == "max" else CNN_POOL_AVG
                d.kernel_h, d.kernel_w = layer.kernel
                d.stride_h, d.stride_w = layer.stride
                d.pad_h, d.pad_w = layer.pad
                d.ceil_mode = int(layer.ceil)
                d.fuse_relu = int(layer.relu)
            elif layer.kind == "lrn":
                d.type = CNN_LAYER_LRN
                d.lrn_size = layer.size
                d.lrn_alpha, d.lrn_beta, d.lrn_k = layer.alpha, layer.beta, layer.k
            elif layer.kind == "relu":
                d.type = CNN_LAYER_RELU
            elif layer.kind == "softmax":
                d.type = CNN_LAYER_SOFTMAX
            else:
                raise ValueError(f"unknown layer kind {layer.kind}")
            d.weight = w.data_ptr() if w is not None else None
            d.bias = b.data_ptr() if b is not None else None
        self._ws: Optional[torch.Tensor] = None
        self._ws_key = None

    def replica(self) -> "Network":
        """A Network over the same device parameters with its own workspace,
        index buffers and graphs, so that a second pass can run concurrently
        on another stream (two passes never share a workspace)."""
        r = Network.__new__(Network)
        r.execution_mode = self.execution_mode
        r._graphs, r._outs = {}, {}
        r.net, r.device, r.weights = self.net, self.device, self.weights
        r.pool_index = self.pool_index
        r.indices = [None] * len(self.net.layers)
        r.descs = (cnn_layer_desc * len(self.descs))()
        ctypes.memmove(r.descs, self.descs, ctypes.sizeof(self.descs))
        for d in r.descs:
            d.pool_index = None
        r._ws, r._ws_key = None, None
        return r

    def out_shape(self, N: int) -> Tuple[int, int, int, int]:
        C, H, W = self.net.input_chw
        oc, oh, ow = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        _ok(lib.cnn_net_out_shape(self.descs, len(self.descs), N, C, H, W, ctypes.byref(oc),
                                  ctypes.byref(oh), ctypes.byref(ow)))
        last = [l for l in self.net.layers if l.kind not in ("relu", "softmax")]
        if last and last[-1].kind == "fc":
            return (N, oc.value)
        return (N, oc.value, oh.value, ow.value)

    def workspace_bytes(self, N: int) -> int:
        C, H, W = self.net.input_chw
        n = lib.cnn_net_workspace_bytes(self.descs, len(self.descs), N, C, H, W)
        if n == 0 and N > 0:
            raise CnnError(CNN_ERR_INVALID, cnn_last_error())
        return int(n)

    @classmethod
    def from_netfile(cls, netfile, params, device="cuda", pool_index: bool = False) -> "Network":
        """A Network for a parsed NetFile (or NetFile text): its execution
        mode, and auto-tuning switched on for the library when it asks so."""
        if isinstance(netfile, str):
            netfile = parse_netfile(netfile)
        if netfile.auto_tuning:
            cnn_set_autotune(True)
        return cls(netfile.net, params, device, pool_index, netfile.execution_mode)

    def close(self) -> None:
        """Destroys the captured graphs."""
        for g in self._graphs.values():
            lib.cnn_net_graph_destroy(g)
        self._graphs.clear()

    def __del__(self):
        try:
            self.close()
        except Exception:  # interpreter shutdown
            pass

    def _prepare(self, N: int):
        key = N
        if self._ws_key != key:
            self.close()  # graphs hold the old workspace and index buffers
            nbytes = self.workspace_bytes(N)
            self._ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
            self._ws_key = key
            if self.pool_index:
                self._alloc_indices(N)

    def _alloc_indices(self, N: int):
        C, H, W = self.net.input_chw
        c, h, w = C, H, W
        for i, layer in enumerate(self.net.layers):
            if layer.kind == "conv":
                h, w = cnn_conv2d_out_shape(h, w, *layer.kernel, layer.stride, layer.pad)
                c = layer.out_channels
            elif layer.kind == "pool":
                h, w = cnn_pool_out_shape(h, w, layer.kernel, layer.stride, layer.pad, layer.ceil)
                if layer.mode == "max":
                    self.indices[i] = torch.empty((N, c, h, w), dtype=torch.int32, device=self.device)
                    self.descs[i].pool_index = self.indices[i].data_ptr()
            elif layer.kind == "fc":
                c, h, w = layer.out_features, 1, 1

    def forward(self, x: torch.Tensor, y: Optional[torch.Tensor] = None, stream=None,
                events: Optional[Sequence] = None,
                kernel_events: Optional[Tuple[Sequence, Sequence]] = None) -> torch.Tensor:
        """cnn_net_fwd; cnn_net_fwd_timed with `events` (one torch.cuda.Event
        per layer + 1); cnn_net_fwd_kernel_timed with `kernel_events` = (starts,
        stops), one event of each per layer, every event already recorded once
        (torch creates its events lazily)."""
        N, C, H, W = x.shape
        self._prepare(N)
        if events is not None and kernel_events is not None:
            raise ValueError("events and kernel_events are exclusive")
        graph = self.execution_mode == "graph" and events is None and kernel_events is None
        if y is None:
            if graph:
                if N not in self._outs:
                    self._outs[N] = torch.empty(self.out_shape(N), dtype=torch.float32, device=x.device)
                y = self._outs[N]
            else:
                y = torch.empty(self.out_shape(N), dtype=torch.float32, device=x.device)
        args = (self.descs, len(self.descs), _dev(x, "x"), N, C, H, W, _dev(y, "y"),
                self._ws.data_ptr(), self._ws.numel())
        if graph:
            key = (N, C, H, W, x.data_ptr(), y.data_ptr())
            g = self._graphs.get(key)
            if g is None:
                # eager first pass: validates, and tunes new shapes when auto-tuning is on
                _ok(lib.cnn_net_fwd(*args, _stream(stream)))
                g = ctypes.c_void_p()
                _ok(lib.cnn_net_graph_create(*args, ctypes.byref(g)))
                self._graphs[key] = g
                return y
            _ok(lib.cnn_net_graph_launch(g, _stream(stream)))
            return y
        if kernel_events is not None:
            starts, stops = kernel_events
            if len(starts) != len(self.descs) or len(stops) != len(self.descs):
                raise ValueError("need one start and one stop event per layer")
            arrs = [(ctypes.c_void_p * len(ev))(*[e.cuda_event if hasattr(e, "cuda_event") else int(e) for e in ev])
                    for ev in (starts, stops)]
            _ok(lib.cnn_net_fwd_kernel_timed(*args, arrs[0], arrs[1], _stream(stream)))
        elif events is None:
            _ok(lib.cnn_net_fwd(*args, _stream(stream)))
        else:
            if len(events) != len(self.descs) + 1:
                raise ValueError("need one event per layer plus one")
            arr = (ctypes.c_void_p * len(events))(*[e.cuda_event if hasattr(e, "cuda_event") else int(e)
                                                    for e in events])
            _ok(lib.cnn_net_fwd_timed(*args, arr, _stream(stream)))
        return y

    __call__ = forward

    def forward_noalloc(self, x: torch.Tensor, y: Optional[torch.Tensor] = None, stream=None):
        """cnn_net_fwd_noalloc: the pass with the library's static device
        scratch as its workspace (no workspace tensor is allocated here; y is
        allocated when None)."""
        N, C, H, W = x.shape
        if y is None:
            y = torch.empty(self.out_shape(N), dtype=torch.float32, device=x.device)
        _ok(lib.cnn_net_fwd_noalloc(self.descs, len(self.descs), _dev(x, "x"), N, C, H, W, _dev(y, "y"),
                                    _stream(stream)))
        return y

    def layer_shapes(self, N: int) -> List[Tuple[int, ...]]:
        """Output shape of every layer for a batch of N (the library's shape rules)."""
        C, H, W = self.net.input_chw
        oc, oh, ow = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        shapes = []
        flat = False  # after an FC layer (and the ReLU / softmax layers after it): [N][O]
        for i, layer in enumerate(self.net.layers):
            _ok(lib.cnn_net_out_shape(self.descs, i + 1, N, C, H, W, ctypes.byref(oc),
                                      ctypes.byref(oh), ctypes.byref(ow)))
            if layer.kind not in ("relu", "softmax"):
                flat = layer.kind == "fc"
            shapes.append((N, oc.value) if flat else (N, oc.value, oh.value, ow.value))
        return shapes

    def forward_dump(self, x: torch.Tensor, y: Optional[torch.Tensor] = None, stream=None):
        """cnn_net_fwd_dump: one pass that also writes every layer's output.

        Returns (y, outs, written): outs[i] is layer i's output (a tensor of
        its shape) where written[i], else None (a RELU layer executed inside
        its predecessor, whose entry then holds the output after it)."""
        N, C, H, W = x.shape
        self._prepare(N)
        if y is None:
            y = torch.empty(self.out_shape(N), dtype=torch.float32, device=x.device)
        bufs = [torch.empty(s, dtype=torch.float32, device=x.device) for s in self.layer_shapes(N)]
        ptrs = (ctypes.c_void_p * len(bufs))(*[b.data_ptr() for b in bufs])
        written = (ctypes.c_int * len(bufs))()
        _ok(lib.cnn_net_fwd_dump(self.descs, len(self.descs), _dev(x, "x"), N, C, H, W, _dev(y, "y"),
                                 self._ws.data_ptr(), self._ws.numel(), ptrs, written, _stream(stream)))
        flags = [bool(written[i]) for i in range(len(bufs))]
        return y, [b if f else None for b, f in zip(bufs, flags)], flags


def cnn_net_fwd(network: Network, x, y=None, stream=None):
    return network.forward(x, y, stream)
