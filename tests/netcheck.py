"""Layer-by-layer comparison of a network pass with the oracle.

A network pass of the HIP path writes every layer's output
(``Network.forward_dump``, the C call ``cnn_net_fwd_dump``).  Each layer i is
checked twice:

  chain  against the oracle's own network on the same input (the oracle's
         layer-i output), with the conv / FC criterion of parity.py:
         max abs error <= 1e-4 * sqrt(Kred) and relative L2 <= 1e-4, where
         Kred is that of the layer itself for conv / FC and of the nearest
         conv / FC layer before it for the layers that only pass values on
         (pooling, LRN, ReLU): a max or mean of values, or LRN's scaling by at
         most 1, does not enlarge an absolute error.
  local  against the oracle's layer i applied to the HIP path's OWN input of
         that layer (the previous layer's dumped output), i.e. on identical
         inputs: conv / FC with the same criterion, max pooling bit-exact in
         values and indices, ReLU bit-exact, average pooling and LRN within
         elementwise relative 1e-5.

Max-pool indices inside a network (the scope table's net-level argmax
rule): the local check already makes them bit-exact on the HIP path's own
input (so each index lies in its window and points at its pooled value).
Against the oracle's chain an index may differ only where the oracle's
window holds a near tie: the oracle's values at the two indices differ by no
more than the upstream absolute tolerance.

A RELU layer executed inside its predecessor has no output of its own: the
predecessor's dump holds the value after that ReLU and is compared with the
oracle's output of the last such RELU layer.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence

import numpy as np

import oracle
from parity import assert_elementwise_close, assert_gemm_close


def _kred(layer, in_shape) -> int:
    if layer.kind == "conv":
        return (layer.in_channels // layer.groups) * layer.kernel[0] * layer.kernel[1]
    if layer.kind == "fc":
        return int(np.prod(in_shape[1:]))
    raise ValueError(layer.kind)


def _oracle_layer(layer, params, x, relu_after: bool):
    """The oracle's layer on x (then a ReLU for a folded RELU layer after it);
    for max pooling also the indices."""
    idx = None
    if layer.kind == "conv":
        y = oracle.conv2d_fwd(x, params[0], params[1], layer.stride, layer.pad, layer.groups, layer.relu)
    elif layer.kind == "fc":
        y = oracle.fc_fwd(x.reshape(x.shape[0], -1), params[0], params[1], layer.relu)
    elif layer.kind == "pool":
        r = oracle.pool_fwd(x, layer.mode, layer.kernel, layer.stride, layer.pad, layer.ceil, layer.relu,
                            with_index=(layer.mode == "max"))
        y, idx = r if isinstance(r, tuple) else (r, None)
    elif layer.kind == "lrn":
        y = oracle.lrn_fwd(x, layer.size, layer.alpha, layer.beta, layer.k)
    elif layer.kind == "relu":
        y = oracle.relu_fwd(x)
    elif layer.kind == "softmax":
        y = oracle.softmax_fwd(x)
    else:
        raise ValueError(layer.kind)
    if relu_after:
        y = oracle.relu_fwd(y)
    return y, idx


def _window_extent(layer, H, W, p, q):
    r0 = p * layer.stride[0] - layer.pad[0]
    c0 = q * layer.stride[1] - layer.pad[1]
    return max(r0, 0), min(r0 + layer.kernel[0], H), max(c0, 0), min(c0 + layer.kernel[1], W)


def check_index_near_ties(layer, x_ref, idx_gpu, idx_ref, atol, what):
    """Net-level argmax rule: where the HIP path's index differs from the
    oracle's, it lies in the window and the oracle's input values at the two
    indices differ by at most atol (a near tie in the oracle's window)."""
    N, C, H, W = x_ref.shape
    assert idx_gpu.shape == idx_ref.shape, (what, idx_gpu.shape, idx_ref.shape)
    assert idx_gpu.min(initial=0) >= 0 and idx_gpu.max(initial=0) < H * W, f"{what}: index out of range"
    diff = np.argwhere(idx_gpu != idx_ref)
    planes = x_ref.reshape(N, C, H * W)
    for n, c, p, q in diff:
        ig, ir = int(idx_gpu[n, c, p, q]), int(idx_ref[n, c, p, q])
        h0, h1, w0, w1 = _window_extent(layer, H, W, p, q)
        assert h0 <= ig // W < h1 and w0 <= ig % W < w1, \
            f"{what}: index {ig} of ({n},{c},{p},{q}) outside its window"
        gap = abs(float(planes[n, c, ig]) - float(planes[n, c, ir]))
        assert gap <= atol, (f"{what}: index {ig} vs oracle {ir} at ({n},{c},{p},{q}) is not a near tie "
                             f"(gap {gap:.3e} > {atol:.3e})")
    return len(diff)


def compare_layers(net, params, x, outs: Sequence[Optional[np.ndarray]], written: Sequence[bool],
                   ref_outs: Sequence[np.ndarray], idx: Optional[Sequence] = None,
                   ref_idx: Optional[Sequence] = None, what: str = "", local: bool = True) -> List[str]:
    """Checks every layer of one pass; raises AssertionError naming the first
    layer that fails.  x: the network input (the sampled images); outs[i]: the
    HIP path's layer-i output on those images (None where not written);
    ref_outs[i]: the oracle's chain output of layer i on them; idx / ref_idx:
    max-pool indices per layer (None elsewhere), optional.  Returns one
    summary line per checked layer."""
    layers = net.layers
    n = len(layers)
    report = []
    kred_up = None          # Kred of the nearest conv / FC layer so far
    gpu_in = x              # the HIP path's input of the current layer
    ref_in = x              # the oracle chain's input of the current layer
    shape_in = x.shape
    i = 0
    while i < n:
        layer = layers[i]
        if not written[i]:
            raise AssertionError(f"{what}: layer {i} ({layer.kind}) has no output and is not a folded ReLU")
        # RELU layers folded into this one
        j = i
        while j + 1 < n and not written[j + 1]:
            assert layers[j + 1].kind == "relu", f"{what}: layer {j + 1} ({layers[j + 1].kind}) not written"
            j += 1
        g = np.asarray(outs[i])
        r = np.asarray(ref_outs[j])
        tag = f"{what} layer {i} ({layer.kind}{'+relu' * (j - i)})"
        if layer.kind in ("conv", "fc"):
            kred_up = _kred(layer, shape_in)
        k = kred_up if kred_up is not None else 1
        # chain
        if layer.kind == "softmax":
            np.testing.assert_allclose(g, r, rtol=1e-4, atol=1e-30, err_msg=f"{tag} chain")
            err = float(np.max(np.abs(g.astype(np.float64) - r), initial=0.0))
        else:
            try:
                err = assert_gemm_close(g, r, k, f"{tag} chain")
            except AssertionError as e:
                raise AssertionError(str(e)) from None
        line = f"{tag}: chain max abs {err:.2e} (tol {1e-4 * math.sqrt(k):.2e})"
        # local: the oracle's layer on the HIP path's own input
        if local:
            lo, lidx = _oracle_layer(layer, params[i] if params is not None else None, np.asarray(gpu_in),
                                     relu_after=j > i)
            if layer.kind in ("conv", "fc"):
                e2 = assert_gemm_close(g, lo, k, f"{tag} local")
                line += f", local max abs {e2:.2e}"
            elif layer.kind == "pool" and layer.mode == "max" or layer.kind == "relu":
                if not np.array_equal(g, lo):
                    bad = int(np.sum(g != lo))
                    raise AssertionError(f"{tag} local: {bad} values differ from the oracle on identical input")
                if layer.kind == "pool" and idx is not None and idx[i] is not None:
                    if not np.array_equal(np.asarray(idx[i]), lidx):
                        bad = int(np.sum(np.asarray(idx[i]) != lidx))
                        raise AssertionError(f"{tag} local: {bad} indices differ from the oracle on identical input")
                line += ", local bit-exact"
            elif layer.kind == "softmax":
                np.testing.assert_allclose(g, lo, rtol=1e-5, atol=1e-30, err_msg=f"{tag} local")
            else:   # avg pool, LRN
                assert_elementwise_close(g, lo, np.abs(np.asarray(gpu_in)).max(initial=0.0), f"{tag} local")
                line += ", local rel 1e-5"
        if layer.kind == "pool" and layer.mode == "max" and idx is not None and ref_idx is not None \
                and idx[i] is not None and ref_idx[i] is not None:
            nd = check_index_near_ties(layer, np.asarray(ref_in), np.asarray(idx[i]), np.asarray(ref_idx[i]),
                                       1e-4 * math.sqrt(k), tag)
            line += f", {nd} of {np.asarray(idx[i]).size} indices differ from the chain (near ties)"
        report.append(line)
        gpu_in, ref_in = g, r
        shape_in = g.shape
        i = j + 1
    return report


def dump_and_compare(gpu, net, params, x, rows=None, model=None, what=None):
    """Runs x through cnn_net_fwd_dump (max-pool indices on) and checks every
    layer of the sampled images `rows` (all when None) with compare_layers.
    The final output must equal the last dump bit for bit, and a plain
    cnn_net_fwd pass must agree with it.  Returns the Network used."""
    import torch

    batch = x.shape[0]
    what = what or f"{net.name} B{batch}"
    if model is None:
        model = gpu.Network(net, params, pool_index=True)
    xd = torch.from_numpy(x).cuda()
    y, outs, written = model.forward_dump(xd)
    rows = list(range(batch)) if rows is None else list(rows)
    torch.cuda.synchronize()
    g = [None if o is None else o[rows].cpu().numpy() for o in outs]
    gi = [None if t is None else t[rows].cpu().numpy() for t in model.indices]
    yh = y.cpu().numpy()
    last = max(i for i, w in enumerate(written) if w)
    np.testing.assert_array_equal(yh[rows].reshape(g[last].shape), g[last])
    y2 = model(xd).cpu().numpy()
    assert_gemm_close(y2[rows].reshape(g[last].shape), g[last], 1, f"{what}: plain pass vs dumped pass")
    _r, ref, ref_idx = oracle.net_fwd(net, x[rows], params, keep=True, pool_index=True)
    rep = compare_layers(net, params, x[rows], g, written, ref, gi, ref_idx, what)
    print("\n".join(rep), flush=True)
    return model
