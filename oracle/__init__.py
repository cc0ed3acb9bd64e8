"""CPU oracle of the CNN forward layers -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It wraps ``liboracle.so`` (plain C,
double accumulation, see ``oracle.h`` for each layer's definition) with numpy
arrays, and composes whole networks layer by layer in the order of the
paper's layer-setup table (Sec. 4): each listed layer runs, then its ReLU if
the table writes "+ReLU".  It shares no code with the GPU path; the only
module both read is ``paper_1511_07376_amd.workloads`` (network descriptions
and seeded generators, no layer arithmetic).
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

_c_int = ctypes.c_int
_fp = ctypes.POINTER(ctypes.c_float)
_ip = ctypes.POINTER(ctypes.c_int32)

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _build  # noqa: WPS433 (build on first use in tests)
        _build.build()
    lib = ctypes.CDLL(LIB_PATH)
    lib.oracle_conv2d_out_shape.argtypes = [_c_int] * 8 + [ctypes.POINTER(_c_int)] * 2
    lib.oracle_pool_out_shape.argtypes = [_c_int] * 9 + [ctypes.POINTER(_c_int)] * 2
    lib.oracle_conv2d_fwd.argtypes = ([_fp] + [_c_int] * 4 + [_fp] + [_c_int] * 3 + [_fp]
                                      + [_c_int] * 6 + [_fp])
    lib.oracle_fc_fwd.argtypes = [_fp, _c_int, _c_int, _fp, _fp, _c_int, _c_int, _fp]
    lib.oracle_pool_fwd.argtypes = [_fp] + [_c_int] * 13 + [_fp, _ip]
    lib.oracle_lrn_fwd.argtypes = [_fp] + [_c_int] * 5 + [ctypes.c_float] * 3 + [_fp]
    lib.oracle_relu_fwd.argtypes = [_fp, _fp, ctypes.c_int64]
    lib.oracle_softmax_fwd.argtypes = [_fp, _c_int, _c_int, _c_int, _fp]
    lib.oracle_set_threads.argtypes = [_c_int]
    lib.oracle_get_threads.restype = _c_int
    for name in ("oracle_conv2d_out_shape", "oracle_pool_out_shape", "oracle_conv2d_fwd",
                 "oracle_fc_fwd", "oracle_pool_fwd", "oracle_lrn_fwd", "oracle_relu_fwd",
                 "oracle_softmax_fwd"):
        getattr(lib, name).restype = _c_int
    _lib = lib
    return lib


def use_library(path: str) -> None:
    """Point the wrappers at another build of oracle.c (the mutation tests use
    this to check that planted mistakes are caught by the pins)."""
    global _lib, LIB_PATH
    _lib = None
    LIB_PATH = path


def _f32(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a


def _ptr(a: Optional[np.ndarray]):
    if a is None:
        return None
    if a.dtype == np.int32:
        return a.ctypes.data_as(_ip)
    return a.ctypes.data_as(_fp)


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise ValueError(f"oracle: {what} rejected its arguments")


def set_threads(n: int) -> None:
    _load().oracle_set_threads(int(n))


def get_threads() -> int:
    return int(_load().oracle_get_threads())


def conv2d_out_shape(H, W, R, S, sh, sw, ph, pw) -> Tuple[int, int]:
    P, Q = _c_int(), _c_int()
    _check(_load().oracle_conv2d_out_shape(H, W, R, S, sh, sw, ph, pw,
                                           ctypes.byref(P), ctypes.byref(Q)), "conv2d_out_shape")
    return P.value, Q.value


def pool_out_shape(H, W, kh, kw, sh, sw, ph, pw, ceil_mode=True) -> Tuple[int, int]:
    P, Q = _c_int(), _c_int()
    _check(_load().oracle_pool_out_shape(H, W, kh, kw, sh, sw, ph, pw, int(ceil_mode),
                                         ctypes.byref(P), ctypes.byref(Q)), "pool_out_shape")
    return P.value, Q.value


def conv2d_fwd(x, w, bias=None, stride=(1, 1), pad=(0, 0), groups=1, relu=False) -> np.ndarray:
    """x [N][C][H][W], w [K][C/G][R][S], bias [K] or None -> y [N][K][P][Q]."""
    x, w = _f32(x), _f32(w)
    bias = None if bias is None else _f32(bias)
    N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if Cg * groups != C:
        raise ValueError("oracle: weight channels do not match input channels / groups")
    P, Q = conv2d_out_shape(H, W, R, S, stride[0], stride[1], pad[0], pad[1])
    y = np.empty((N, K, P, Q), np.float32)
    _check(_load().oracle_conv2d_fwd(_ptr(x), N, C, H, W, _ptr(w), K, R, S, _ptr(bias),
                                     stride[0], stride[1], pad[0], pad[1], groups,
                                     int(relu), _ptr(y)), "conv2d_fwd")
    return y


def fc_fwd(x, w, bias=None, relu=False) -> np.ndarray:
    """x [N][I] (or any [N][...] flattened in C order), w [O][I] -> y [N][O]."""
    x = _f32(x).reshape(x.shape[0], -1)
    w = _f32(w)
    bias = None if bias is None else _f32(bias)
    N, I = x.shape
    O, I2 = w.shape
    if I2 != I:
        raise ValueError(f"oracle: fc expects {I2} inputs, got {I}")
    y = np.empty((N, O), np.float32)
    _check(_load().oracle_fc_fwd(_ptr(x), N, I, _ptr(w), _ptr(bias), O, int(relu), _ptr(y)),
           "fc_fwd")
    return y


def pool_fwd(x, mode="max", kernel=(2, 2), stride=(2, 2), pad=(0, 0), ceil_mode=True,
             relu=False, with_index=False):
    """mode "max" or "avg".  Returns y, or (y, idx) for max with with_index."""
    x = _f32(x)
    N, C, H, W = x.shape
    P, Q = pool_out_shape(H, W, kernel[0], kernel[1], stride[0], stride[1], pad[0], pad[1],
                          ceil_mode)
    y = np.empty((N, C, P, Q), np.float32)
    idx = np.empty((N, C, P, Q), np.int32) if (mode == "max" and with_index) else None
    m = {"max": 0, "avg": 1}[mode]
    _check(_load().oracle_pool_fwd(_ptr(x), N, C, H, W, m, kernel[0], kernel[1], stride[0],
                                   stride[1], pad[0], pad[1], int(ceil_mode), int(relu),
                                   _ptr(y), _ptr(idx)), "pool_fwd")
    return (y, idx) if idx is not None else y


def lrn_fwd(x, size=5, alpha=1e-4, beta=0.75, k=1.0) -> np.ndarray:
    x = _f32(x)
    N, C, H, W = x.shape
    y = np.empty_like(x)
    _check(_load().oracle_lrn_fwd(_ptr(x), N, C, H, W, size, alpha, beta, k, _ptr(y)),
           "lrn_fwd")
    return y


def relu_fwd(x) -> np.ndarray:
    x = _f32(x)
    y = np.empty_like(x)
    _check(_load().oracle_relu_fwd(_ptr(x), _ptr(y), x.size), "relu_fwd")
    return y


def softmax_fwd(x) -> np.ndarray:
    """Softmax across axis 1 of an [N][C] or [N][C][H][W] array."""
    x = _f32(x)
    if x.ndim < 2:
        raise ValueError("oracle: softmax needs an [N][C...] array")
    N, C = x.shape[0], x.shape[1]
    HW = int(np.prod(x.shape[2:])) if x.ndim > 2 else 1
    y = np.empty_like(x)
    _check(_load().oracle_softmax_fwd(_ptr(x), N, C, HW, _ptr(y)), "softmax_fwd")
    return y


def net_fwd(net, x, params, keep: bool = False, pool_index: bool = False):
    """Run a ``workloads.Net`` on input x with ``workloads.make_params`` params.

    Each layer runs as written in the layer list, followed by a separate ReLU
    where the layer carries one.  Returns the final output; with ``keep``, also
    the list of every layer's output, and with ``pool_index`` also the list of
    max-pool indices (None for other layers).
    """
    outs: List[np.ndarray] = []
    idxs: List[Optional[np.ndarray]] = []
    a = _f32(x)
    for layer, pr in zip(net.layers, params):
        ix = None
        if layer.kind == "conv":
            if a.shape[1] != layer.in_channels:
                raise ValueError("oracle: conv input channels mismatch")
            a = conv2d_fwd(a, pr[0], pr[1], layer.stride, layer.pad, layer.groups)
        elif layer.kind == "fc":
            flat = a.reshape(a.shape[0], -1)
            if flat.shape[1] != layer.in_features:
                raise ValueError(f"oracle: fc expects {layer.in_features} features, "
                                 f"got {flat.shape[1]}")
            a = fc_fwd(flat, pr[0], pr[1])
        elif layer.kind == "pool":
            r = pool_fwd(a, layer.mode, layer.kernel, layer.stride, layer.pad, layer.ceil,
                         with_index=(pool_index and layer.mode == "max"))
            if isinstance(r, tuple):
                a, ix = r
            else:
                a = r
        elif layer.kind == "lrn":
            a = lrn_fwd(a, layer.size, layer.alpha, layer.beta, layer.k)
        elif layer.kind == "relu":
            a = relu_fwd(a)
        elif layer.kind == "softmax":
            a = softmax_fwd(a)
        else:
            raise ValueError(f"oracle: unknown layer kind {layer.kind}")
        if layer.relu and layer.kind != "relu":
            a = relu_fwd(a)
        outs.append(a)
        idxs.append(ix)
    if keep and pool_index:
        return a, outs, idxs
    if keep:
        return a, outs
    if pool_index:
        return a, idxs
    return a
