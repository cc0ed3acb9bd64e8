"""Seeded synthetic workloads shaped like the paper's benchmark networks.

The paper evaluates three networks, LeNet for MNIST, Alex Krizhevsky's CIFAR-10
network and AlexNet for ImageNet 2012 (Sec. 4, layer-setup table), on batches
of 16 images.  None of the datasets or trained models are used here: every
input image and every parameter is drawn from a seeded generator with the
shapes of those networks.

This module describes inputs only.  It lists each network's layers with their
hyper-parameters (including the channel and feature counts each parameterised
layer expects, so that parameter shapes need no layer arithmetic) and draws the
seeded tensors.  It holds none of the layers' arithmetic, which is why both the
HIP path and the CPU oracle may read it.

Seeds: tensor ``t`` of a run with base seed ``s`` is drawn from
``numpy.random.default_rng(1000 * s + t)`` (PCG64).  Tensor ids are given in
layer order: the input batch is 0, then weight and bias of each parameterised
layer.  Values are drawn in float64 and rounded to float32 once; the same
float32 bytes go to the oracle and to the GPU.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

__all__ = [
    "Layer", "Net", "conv", "fc", "pool", "lrn", "relu", "softmax",
    "NETS", "lenet", "cifar_quick", "alexnet", "alexnet_he",
    "SWEEP_SHAPES", "SWEEP_BATCHES",
    "rng_for", "uniform01", "normal", "make_input", "make_params",
    "make_sweep_tensors",
]


@dataclass(frozen=True)
class Layer:
    """One layer of a network description.

    kind: "conv", "fc", "pool", "lrn", "relu" or "softmax" (across channels).
    conv: in_channels, out_channels, kernel (R, S), stride, pad, groups, relu.
    fc:   in_features, out_features, relu.
    pool: mode ("max" or "avg"), kernel, stride, pad, ceil, relu (applied
          after pooling, as the paper's "Pooling+ReLU" row).
    lrn:  size, alpha, beta, k.
    """

    kind: str
    in_channels: int = 0
    out_channels: int = 0
    kernel: Tuple[int, int] = (1, 1)
    stride: Tuple[int, int] = (1, 1)
    pad: Tuple[int, int] = (0, 0)
    groups: int = 1
    relu: bool = False
    in_features: int = 0
    out_features: int = 0
    mode: str = "max"
    ceil: bool = True
    size: int = 5
    alpha: float = 1e-4
    beta: float = 0.75
    k: float = 1.0

    @property
    def has_params(self) -> bool:
        return self.kind in ("conv", "fc")

    def weight_shape(self) -> Tuple[int, ...]:
        if self.kind == "conv":
            return (self.out_channels, self.in_channels // self.groups,
                    self.kernel[0], self.kernel[1])
        if self.kind == "fc":
            return (self.out_features, self.in_features)
        raise ValueError(f"{self.kind} layer has no weights")

    def bias_shape(self) -> Tuple[int, ...]:
        if self.kind == "conv":
            return (self.out_channels,)
        if self.kind == "fc":
            return (self.out_features,)
        raise ValueError(f"{self.kind} layer has no bias")


def _pair(v) -> Tuple[int, int]:
    return (v, v) if isinstance(v, int) else (int(v[0]), int(v[1]))


def conv(cin: int, cout: int, k, stride=1, pad=0, groups: int = 1,
         relu: bool = False) -> Layer:
    return Layer("conv", in_channels=cin, out_channels=cout, kernel=_pair(k),
                 stride=_pair(stride), pad=_pair(pad), groups=groups, relu=relu)


def fc(fin: int, fout: int, relu: bool = False) -> Layer:
    return Layer("fc", in_features=fin, out_features=fout, relu=relu)


def pool(mode: str, k, stride, pad=0, ceil: bool = True, relu: bool = False) -> Layer:
    assert mode in ("max", "avg")
    return Layer("pool", mode=mode, kernel=_pair(k), stride=_pair(stride),
                 pad=_pair(pad), ceil=ceil, relu=relu)


def lrn(size: int = 5, alpha: float = 1e-4, beta: float = 0.75, k: float = 1.0) -> Layer:
    return Layer("lrn", size=size, alpha=alpha, beta=beta, k=k)


def relu() -> Layer:
    return Layer("relu")


def softmax() -> Layer:
    return Layer("softmax")


@dataclass(frozen=True)
class Net:
    """A network description: input image shape (C, H, W), layers in order,
    the standard deviations of the N(0, std) weights and biases, the input
    distribution ("uniform01" or "normal") and the paper's batch size.

    weight_init "he" replaces weight_std by sqrt(2 / fan_in) per layer (fan_in
    = the product of a weight tensor's dimensions after the first), and
    input_scale multiplies the drawn input."""

    name: str
    input_chw: Tuple[int, int, int]
    layers: Tuple[Layer, ...]
    weight_std: float
    bias_std: float
    input_dist: str = "uniform01"
    default_batch: int = 16
    batches: Tuple[int, ...] = field(default_factory=tuple)
    weight_init: str = "normal"
    input_scale: float = 1.0


# Layer order and fusion points follow the paper's layer-setup table (Sec. 4):
# LeNet: Conv, Pooling, Conv, Pooling, FC+ReLU, FC.
lenet = Net(
    name="lenet",
    input_chw=(1, 28, 28),
    layers=(
        conv(1, 20, 5),
        pool("max", 2, 2),
        conv(20, 50, 5),
        pool("max", 2, 2),
        fc(800, 500, relu=True),
        fc(500, 10),
    ),
    weight_std=0.05, bias_std=0.01, default_batch=16, batches=(16,),
)

# Alex's CIFAR-10: Conv, Pooling+ReLU, Conv+ReLU, Pooling, Conv+ReLU, Pooling,
# FC, FC.  The first pooling is max, the other two average (CIFAR-10 "quick").
cifar_quick = Net(
    name="cifar_quick",
    input_chw=(3, 32, 32),
    layers=(
        conv(3, 32, 5, pad=2),
        pool("max", 3, 2, relu=True),
        conv(32, 32, 5, pad=2, relu=True),
        pool("avg", 3, 2),
        conv(32, 64, 5, pad=2, relu=True),
        pool("avg", 3, 2),
        fc(1024, 64),
        fc(64, 10),
    ),
    weight_std=0.05, bias_std=0.01, default_batch=32, batches=(32,),
)

# AlexNet: Conv+ReLU, LRN, Pooling, Conv+ReLU, LRN, Pooling, Conv+ReLU,
# Conv+ReLU, Conv+ReLU, Pooling, FC+ReLU, FC+ReLU, FC.
alexnet = Net(
    name="alexnet",
    input_chw=(3, 227, 227),
    layers=(
        conv(3, 96, 11, stride=4, relu=True),
        lrn(5, 1e-4, 0.75, 1.0),
        pool("max", 3, 2),
        conv(96, 256, 5, pad=2, groups=2, relu=True),
        lrn(5, 1e-4, 0.75, 1.0),
        pool("max", 3, 2),
        conv(256, 384, 3, pad=1, relu=True),
        conv(384, 384, 3, pad=1, groups=2, relu=True),
        conv(384, 256, 3, pad=1, groups=2, relu=True),
        pool("max", 3, 2),
        fc(9216, 4096, relu=True),
        fc(4096, 4096, relu=True),
        fc(4096, 1000),
    ),
    weight_std=0.01, bias_std=0.01, default_batch=16, batches=(16, 64, 256),
)

NETS: Dict[str, Net] = {n.name: n for n in (lenet, cifar_quick, alexnet)}

# The AlexNet layers with weights drawn at N(0, sqrt(2 / fan_in)) and inputs
# uniform in [0, 8), for parity checks only.  With the benchmark's N(0, 0.01)
# weights the activations shrink layer by layer and the LRN layers change
# their inputs by about 1e-6 relative, far below the comparison tolerance;
# here activations stay between ~4 and ~60 through the whole network, so each
# LRN layer changes its output by 1e-3 to 1e-2 relative and every layer's
# result reaches the last layer's output.
alexnet_he = Net(
    name="alexnet_he", input_chw=alexnet.input_chw, layers=alexnet.layers,
    weight_std=0.0, bias_std=0.01, default_batch=16, batches=(16, 64, 256),
    weight_init="he", input_scale=8.0,
)

# Single-layer conv sweep: (C, H, W, K, R, S, stride, pad), bias + ReLU fused,
# N(0, 1) input, weights and bias.
SWEEP_SHAPES: Tuple[Tuple[int, int, int, int, int, int, int, int], ...] = (
    (3, 224, 224, 64, 7, 7, 2, 3),
    (64, 56, 56, 64, 3, 3, 1, 1),
    (256, 28, 28, 256, 3, 3, 1, 1),
    (512, 14, 14, 512, 3, 3, 1, 1),
    (256, 56, 56, 64, 1, 1, 1, 0),
)
SWEEP_BATCHES: Tuple[int, ...] = (1, 16, 64)


def rng_for(base_seed: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng(1000 * int(base_seed) + int(tensor_id))


def uniform01(shape, base_seed: int, tensor_id: int) -> np.ndarray:
    return rng_for(base_seed, tensor_id).random(shape).astype(np.float32)


def normal(shape, std: float, base_seed: int, tensor_id: int) -> np.ndarray:
    return (rng_for(base_seed, tensor_id).standard_normal(shape) * std).astype(np.float32)


def make_input(net: Net, batch: int, base_seed: int = 0) -> np.ndarray:
    shape = (batch,) + tuple(net.input_chw)
    if net.input_dist == "uniform01":
        x = uniform01(shape, base_seed, 0)
    else:
        x = normal(shape, 1.0, base_seed, 0)
    if net.input_scale != 1.0:
        x = (x * np.float32(net.input_scale)).astype(np.float32)
    return x


def make_params(net: Net, base_seed: int = 0) -> List[Optional[Tuple[np.ndarray, np.ndarray]]]:
    """Per layer: (weight, bias) float32 arrays for conv/fc, None otherwise."""
    out: List[Optional[Tuple[np.ndarray, np.ndarray]]] = []
    tid = 1
    for layer in net.layers:
        if layer.has_params:
            std = net.weight_std
            if net.weight_init == "he":
                std = float(np.sqrt(2.0 / np.prod(layer.weight_shape()[1:])))
            w = normal(layer.weight_shape(), std, base_seed, tid)
            b = normal(layer.bias_shape(), net.bias_std, base_seed, tid + 1)
            out.append((w, b))
            tid += 2
        else:
            out.append(None)
    return out


def make_sweep_tensors(shape, batch: int, base_seed: int = 0):
    """x [N][C][H][W], w [K][C][R][S], b [K], all N(0, 1) float32."""
    c, h, w_, k, r, s, _stride, _pad = shape
    x = normal((batch, c, h, w_), 1.0, base_seed, 0)
    w = normal((k, c, r, s), 1.0, base_seed, 1)
    b = normal((k,), 1.0, base_seed, 2)
    return x, w, b
