"""Randomised network parity (GPU): seeded random layer chains run through
cnn_net_fwd and through the oracle's layer-by-layer network.

The fixed networks exercise the paper's three layer setups; these chains
exercise the network executor's choices on shapes nobody picked by hand:
convolution gather modes (padded, unpadded, strided, grouped), LRN followed
by pooling (fused), ReLU layers run inside their producer, a ReLU left to
the next layer after a split reduction, the pass's bias fills run inside a
pooling kernel, FC chains, a softmax at the end, and batches of 1 (every
conv and FC layer split across workgroups), 5 and 33 (FC tile geometries on
both sides of 32 images).

Each pass runs through cnn_net_fwd_dump and every layer is checked
(tests/netcheck.py): against the oracle's chain and against the oracle's
layer on the pass's own input of that layer, max-pool indices included.
"""
import numpy as np
import pytest

import oracle
from conftest import to_dev, to_host
from paper_1511_07376_amd import workloads as wl
from netcheck import dump_and_compare
from parity import assert_gemm_close

N_NETS = 24
BATCHES = (1, 5, 33)


def random_net(seed: int) -> wl.Net:
    """A chain of 2-6 body layers (conv, pool, LRN, ReLU) on a small input,
    then one or two FC layers and, for odd seeds, a softmax."""
    rng = np.random.default_rng(7000 + seed)
    c = int(rng.choice([1, 3, 4, 8]))
    h = w = int(rng.integers(9, 21))
    chw = (c, h, w)
    layers = []
    n_body = int(rng.integers(2, 7))
    while len(layers) < n_body:
        kind = rng.choice(["conv", "conv", "pool", "lrn", "relu"])
        if kind == "conv":
            k = int(rng.choice([1, 3, 5]))
            if k > h + 2 * (k // 2) or k > w + 2 * (k // 2):
                continue
            stride = int(rng.choice([1, 1, 2]))
            pad = int(rng.integers(0, k // 2 + 1))
            cout = int(rng.choice([4, 8, 12, 16]))
            groups = 2 if (c % 2 == 0 and cout % 2 == 0 and rng.random() < 0.3) else 1
            try:
                oh, ow = oracle.conv2d_out_shape(h, w, k, k, stride, stride, pad, pad)
            except ValueError:  # no output pixel
                continue
            layers.append(wl.conv(c, cout, k, stride, pad, groups, relu=bool(rng.random() < 0.6)))
            c, h, w = cout, oh, ow
        elif kind == "pool":
            k = int(rng.choice([2, 3]))
            if k > h or k > w:
                continue
            stride = int(rng.choice([1, 2]))
            pad = int(rng.integers(0, 2)) if k == 3 else 0
            try:
                oh, ow = oracle.pool_out_shape(h, w, k, k, stride, stride, pad, pad)
            except ValueError:
                continue
            layers.append(wl.pool(str(rng.choice(["max", "avg"])), k, stride, pad,
                                  relu=bool(rng.random() < 0.3)))
            h, w = oh, ow
        elif kind == "lrn":
            layers.append(wl.lrn(int(rng.choice([3, 5])), 1e-2, 0.75, 2.0))
            if h >= 3 and w >= 3 and rng.random() < 0.6:  # LRN then pooling: run fused
                oh, ow = oracle.pool_out_shape(h, w, 3, 3, 2, 2, 0, 0)
                layers.append(wl.pool("max", 3, 2))
                h, w = oh, ow
        else:
            layers.append(wl.relu())
    fin = c * h * w
    if rng.random() < 0.5:
        mid = int(rng.choice([24, 40]))
        layers.append(wl.fc(fin, mid, relu=True))
        fin = mid
    layers.append(wl.fc(fin, 10))
    if seed % 2:
        layers.append(wl.softmax())
    return wl.Net(f"random{seed}", chw, tuple(layers), 0.15, 0.05, input_dist="normal")


def _last_fc_in(net: wl.Net) -> int:
    return [l for l in net.layers if l.kind == "fc"][-1].in_features


def test_random_nets_are_valid():
    """The generator's shape bookkeeping agrees with the oracle network (CPU)."""
    for seed in range(N_NETS):
        net = random_net(seed)
        x = wl.make_input(net, 1, seed)
        y = oracle.net_fwd(net, x, wl.make_params(net, seed))
        assert y.shape == (1, 10) or y.shape == (1, 10, 1, 1), (seed, y.shape)


@pytest.mark.gpu
@pytest.mark.parametrize("seed", range(N_NETS))
def test_random_net_matches_oracle(gpu, seed):
    net = random_net(seed)
    params = wl.make_params(net, seed)
    model = gpu.Network(net, params, pool_index=True)
    kinds = " ".join(l.kind for l in net.layers)
    for batch in BATCHES:
        print(f"random net {seed} ({net.input_chw}: {kinds}) batch {batch}", flush=True)
        x = wl.make_input(net, batch, 100 + seed)
        dump_and_compare(gpu, net, params, x, model=model, what=f"random{seed} B{batch}")


@pytest.mark.gpu
@pytest.mark.parametrize("seed", range(0, N_NETS, 4))
def test_random_net_graph_mode(gpu, seed):
    """The library's graph execution mode (capture once, replay) on random
    chains: every replay, with new input data in the same buffer, matches the
    eager network."""
    net = random_net(seed)
    params = wl.make_params(net, seed)
    eager = gpu.Network(net, params)
    graphed = gpu.Network(net, params, execution_mode="graph")
    x = to_dev(wl.make_input(net, 5, 200 + seed))
    for i in range(3):
        print(f"random net {seed} graph replay {i}", flush=True)
        x.copy_(to_dev(wl.make_input(net, 5, 300 + seed + i)))
        y = to_host(graphed(x))
        ref = to_host(eager(x))
        assert_gemm_close(y, ref, _last_fc_in(net), f"random{seed} graph replay {i}")
    graphed.close()
