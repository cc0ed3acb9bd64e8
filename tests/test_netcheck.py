"""The layer-by-layer network comparison (tests/netcheck.py) on the CPU: it
accepts the oracle's own layer outputs and rejects plausible mistakes of a
network executor (an LRN layer skipped, a wrong max-pool index, a slightly
wrong weight), here planted in the oracle's outputs."""
import dataclasses

import numpy as np
import pytest

import oracle
from netcheck import check_index_near_ties, compare_layers
from paper_1511_07376_amd import workloads as wl


def _chain(net, x, params):
    _y, outs, idxs = oracle.net_fwd(net, x, params, keep=True, pool_index=True)
    return outs, idxs


def _without_lrn(net, x, params):
    """Layer outputs of the network with every LRN layer replaced by the
    identity (what an executor that skips them would produce)."""
    keep = [i for i, l in enumerate(net.layers) if l.kind != "lrn"]
    cut = dataclasses.replace(net, layers=tuple(net.layers[i] for i in keep))
    _y, outs, idxs = oracle.net_fwd(cut, x, [params[i] for i in keep], keep=True, pool_index=True)
    full, fidx, k = [], [], 0
    for i, l in enumerate(net.layers):
        if l.kind == "lrn":
            full.append(full[-1])
            fidx.append(None)
        else:
            full.append(outs[k])
            fidx.append(idxs[k])
            k += 1
    return full, fidx


@pytest.fixture(scope="module")
def alexnet_he_case():
    net = wl.alexnet_he
    x = wl.make_input(net, 1, 0)
    params = wl.make_params(net, 0)
    outs, idxs = _chain(net, x, params)
    return net, x, params, outs, idxs


def test_accepts_the_oracles_own_outputs(alexnet_he_case):
    net, x, params, outs, idxs = alexnet_he_case
    rep = compare_layers(net, params, x, outs, [True] * len(outs), outs, idxs, idxs, "oracle")
    assert len(rep) == len(net.layers)


def test_accepts_folded_relu_layers():
    net = wl.Net("folded", (3, 12, 12), (wl.conv(3, 8, 3, pad=1), wl.relu(), wl.pool("max", 2, 2),
                                        wl.fc(8 * 6 * 6, 5), wl.relu()), 0.3, 0.1, input_dist="normal")
    x = wl.make_input(net, 2, 1)
    params = wl.make_params(net, 1)
    outs, idxs = _chain(net, x, params)
    # an executor that runs each ReLU inside the layer before it: the layer's
    # own output is the value after the ReLU, the RELU layer has none
    dumps = [outs[1], None, outs[2], outs[4], None]
    rep = compare_layers(net, params, x, dumps, [True, False, True, True, False], outs, idxs, idxs, "folded")
    assert len(rep) == 3


@pytest.mark.parametrize("drop", ["both", "lrn2"])
def test_rejects_a_skipped_lrn_layer(alexnet_he_case, drop):
    net, x, params, outs, idxs = alexnet_he_case
    if drop == "both":
        bad, bidx = _without_lrn(net, x, params)
        first = 1
    else:
        # only the second LRN skipped: layers 0-3 as computed, then from the
        # second LRN's input on without it
        cut = dataclasses.replace(net, layers=net.layers[5:])
        tail = oracle.net_fwd(cut, outs[3], params[5:], keep=True, pool_index=True)
        bad = outs[:4] + [outs[3]] + tail[1]
        bidx = idxs[:4] + [None] + tail[2]
        first = 4
    for local in (True, False):
        with pytest.raises(AssertionError, match=f"layer {first} \\(lrn\\)"):
            compare_layers(net, params, x, bad, [True] * len(bad), outs, bidx, idxs, "no lrn", local=local)


def test_benchmark_weights_cannot_see_the_lrn_layers():
    """Why the He-scaled variant exists: with the benchmark's N(0, 0.01)
    weights, skipping both LRN layers changes every layer's output by less
    than the comparison tolerance."""
    net = wl.alexnet
    x = wl.make_input(net, 1, 0)
    params = wl.make_params(net, 0)
    outs, _ = _chain(net, x, params)
    bad, _ = _without_lrn(net, x, params)
    rel = max(np.linalg.norm(a.astype(np.float64) - b) / np.linalg.norm(b) for a, b in zip(bad, outs))
    assert rel < 1e-4


def test_rejects_a_small_weight_error(alexnet_he_case):
    """0.1% too large conv3 weights: caught at conv3 and still visible in the
    last layer's output."""
    net, x, params, outs, idxs = alexnet_he_case
    p2 = list(params)
    p2[6] = ((params[6][0] * np.float32(1.001)).astype(np.float32), params[6][1])
    bad, bidx = _chain(net, x, p2)
    with pytest.raises(AssertionError, match="layer 6 \\(conv\\)"):
        compare_layers(net, params, x, bad, [True] * len(bad), outs, bidx, idxs, "conv3 weights", local=False)
    rel = np.linalg.norm(bad[-1].astype(np.float64) - outs[-1]) / np.linalg.norm(outs[-1])
    assert rel > 1e-4


def test_rejects_a_wrong_pool_index(alexnet_he_case):
    net, x, params, outs, idxs = alexnet_he_case
    bidx = list(idxs)
    wrong = idxs[2].copy()
    n, c, p, q = 0, 5, 3, 4
    wrong[n, c, p, q] += 1          # the next column: inside the window, not the maximum
    bidx[2] = wrong
    with pytest.raises(AssertionError, match="layer 2 \\(pool\\)"):
        compare_layers(net, params, x, outs, [True] * len(outs), outs, bidx, idxs, "index")


def test_index_rule_allows_near_ties_only():
    layer = wl.pool("max", 3, 2)
    x = np.zeros((1, 1, 5, 5), np.float32)
    x[0, 0, 0, 0] = 1.0
    x[0, 0, 0, 1] = 1.0 - 1e-6      # a near tie in window (0, 0)
    x[0, 0, 2, 4] = 3.0
    x[0, 0, 4, 4] = 2.0
    _y, ref = oracle.pool_fwd(x, "max", (3, 3), (2, 2), (0, 0), True, with_index=True)
    gpu = ref.copy()
    gpu[0, 0, 0, 0] = 1             # the near-tied element
    assert check_index_near_ties(layer, x, gpu, ref, 1e-4, "tie") == 1
    gpu = ref.copy()
    gpu[0, 0, 1, 1] = 4 * 5 + 4     # 2.0 against the window's 3.0
    with pytest.raises(AssertionError, match="not a near tie"):
        check_index_near_ties(layer, x, gpu, ref, 1e-4, "no tie")
    gpu = ref.copy()
    gpu[0, 0, 0, 0] = 3             # outside window (0, 0)
    with pytest.raises(AssertionError, match="outside its window"):
        check_index_near_ties(layer, x, gpu, ref, 1e-4, "window")
    gpu[0, 0, 0, 0] = 25
    with pytest.raises(AssertionError, match="out of range"):
        check_index_near_ties(layer, x, gpu, ref, 1e-4, "range")
