"""Network parity: cnn_net_fwd against the oracle's layer-by-layer network on
the same seeded input and parameters (GPU).

The paper checks its library by comparing the last layer's output with
Caffe's on the same input (Sec. 4.1).  Here every layer is compared: the
pass runs through cnn_net_fwd_dump, which also writes each layer's output,
and tests/netcheck.py checks each layer against the oracle's chain and
against the oracle's layer on the HIP path's own input of that layer
(max-pool values and indices bit-exact there; against the chain an index may
differ only at a near tie of the oracle's window).  LeNet (batch 16) and
CIFAR-10 quick (batch 32) run whole on both sides.  For AlexNet the GPU runs
the whole batch (16, 64 and 256, the configurations the benchmark times) and
the oracle sampled images; AlexNet runs both with the benchmark's N(0, 0.01)
weights and with He-scaled weights and larger inputs (workloads.alexnet_he),
under which every layer, the LRN layers included, visibly reaches the output.
"""
import numpy as np
import pytest
import torch

import oracle
from conftest import to_dev, to_host
from netcheck import check_index_near_ties, compare_layers, dump_and_compare
from paper_1511_07376_amd import workloads as wl
from parity import assert_gemm_close

pytestmark = pytest.mark.gpu


def run_layers(gpu, net, batch, sample, seed=0, model=None):
    print(f"net layers {net.name} batch {batch} seed {seed} sample {sample}", flush=True)
    x = wl.make_input(net, batch, seed)
    return dump_and_compare(gpu, net, wl.make_params(net, seed), x, sample, model)


def test_lenet_b16(gpu):
    run_layers(gpu, wl.lenet, 16, None)


def test_cifar_quick_b32(gpu):
    run_layers(gpu, wl.cifar_quick, 32, None)


def test_cifar_quick_b32_seed1(gpu):
    run_layers(gpu, wl.cifar_quick, 32, None, seed=1)


@pytest.mark.parametrize("net", [wl.alexnet, wl.alexnet_he], ids=lambda n: n.name)
@pytest.mark.parametrize("batch,sample", [(16, [0, 15]), (64, [0, 63]), (256, [0, 255])],
                         ids=["b16", "b64", "b256"])
def test_alexnet(gpu, net, batch, sample):
    run_layers(gpu, net, batch, sample)


@pytest.mark.parametrize("net", [wl.alexnet, wl.alexnet_he], ids=lambda n: n.name)
def test_alexnet_b64_tuned_as_benchmarked(gpu, net):
    """The benchmark's procedure: auto-tuning on for a first pass at batch 64
    (each conv shape times every tile configuration and keeps the fastest),
    then passes with the recorded choices; every layer checked on images of
    the tuned pass."""
    params = wl.make_params(net, 0)
    model = gpu.Network(net, params, pool_index=True)
    x = to_dev(wl.make_input(net, 64, 0))
    gpu.cnn_tuning_clear()
    try:
        gpu.cnn_set_autotune(True)
        model(x)
        gpu.cnn_set_autotune(False)
        print("tuned:", gpu.cnn_tuning_export().replace("\n", "; "), flush=True)
        run_layers(gpu, net, 64, [0, 31, 63], model=model)
    finally:
        gpu.cnn_set_autotune(False)
        gpu.cnn_tuning_clear()


def test_lenet_pool_indices_valid(gpu):
    """With indices requested, each max-pool index lies in its window and
    points at its pooled value in the network's own pooling input (bit-exact
    against the oracle's pooling of that input), and differs from the
    oracle's chain only at near ties."""
    run_layers(gpu, wl.lenet, 16, None, seed=2)


def test_timed_forward_matches_and_orders_events(gpu):
    net = wl.cifar_quick
    x = wl.make_input(net, 32, 3)
    params = wl.make_params(net, 3)
    model = gpu.Network(net, params)
    xd = to_dev(x)
    y0 = to_host(model(xd))
    events = [torch.cuda.Event(enable_timing=True) for _ in range(len(net.layers) + 1)]
    for e in events:
        e.record()   # creates the event
    y1 = to_host(model(xd, events=events))
    times = [events[i].elapsed_time(events[i + 1]) for i in range(len(net.layers))]
    assert all(t >= 0 for t in times)
    assert_gemm_close(y1, y0, 64, "timed vs untimed")


def kernel_timed_pass(model, xd, nl):
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(nl)]
    stops = [torch.cuda.Event(enable_timing=True) for _ in range(nl)]
    for e in starts + stops:
        e.record()   # creates the event
    y = model(xd, kernel_events=(starts, stops))
    torch.cuda.synchronize()
    return y, starts, stops


@pytest.mark.parametrize("name,batch", [("cifar_quick", 32), ("alexnet", 16), ("alexnet", 1)])
def test_kernel_timed_forward_matches_and_orders_spans(gpu, name, batch):
    """cnn_net_fwd_kernel_timed: the same output as the untimed pass; every
    layer's span is non-negative, and the span of a layer with kernels ends
    before that of the next layer with kernels begins; a layer executed inside
    another one has an interval of about zero, recorded after the pass's last
    kernel."""
    net = wl.NETS[name]
    print(f"kernel-timed {name} batch {batch}", flush=True)
    x = wl.make_input(net, batch, 4)
    model = gpu.Network(net, wl.make_params(net, 4))
    xd = to_dev(x)
    y0 = to_host(model(xd))
    nl = len(net.layers)
    y1, starts, stops = kernel_timed_pass(model, xd, nl)
    assert_gemm_close(to_host(y1), y0, 64, "kernel-timed vs untimed")
    span = [starts[i].elapsed_time(stops[i]) for i in range(nl)]
    assert all(t >= 0 for t in span), span
    folded = [i for i, layer in enumerate(net.layers)
              if layer.kind == "relu" or (layer.kind == "lrn" and i + 1 < nl and net.layers[i + 1].kind == "pool")]
    kern = [i for i in range(nl) if i not in folded]
    for i, layer in enumerate(net.layers):
        if layer.kind == "conv":
            assert span[i] > 0, (i, span)
    gaps = [stops[a].elapsed_time(starts[b]) for a, b in zip(kern, kern[1:])]
    assert all(g >= 0 for g in gaps), gaps
    last = kern[-1]
    for i in folded:
        assert span[i] < 0.05, (i, span[i])
        assert stops[last].elapsed_time(starts[i]) >= 0, i   # recorded after the last kernel
    total = starts[kern[0]].elapsed_time(stops[last])
    assert sum(span[i] for i in kern) <= total + 1e-3


def test_kernel_timed_empty_batch_records_every_span(gpu):
    """An empty batch launches nothing but still records both events of every
    layer (intervals of about zero), like the timed pass's other contract."""
    net = wl.cifar_quick
    model = gpu.Network(net, wl.make_params(net, 6))
    x = torch.empty((0,) + tuple(net.input_chw), device="cuda")
    y, starts, stops = kernel_timed_pass(model, x, len(net.layers))
    assert y.shape[0] == 0
    for a, b in zip(starts, stops):
        assert 0 <= a.elapsed_time(b) < 0.05


def test_kernel_timed_span_leaves_out_autotuning(gpu):
    """A conv layer tuned during a kernel-timed pass counts only its final
    launch: its span is of the order of the same layer's span once tuned, not
    of the candidates' runs."""
    net = wl.lenet
    x = wl.make_input(net, 16, 5)
    model = gpu.Network(net, wl.make_params(net, 5))
    xd = to_dev(x)
    nl = len(net.layers)
    gpu.cnn_tuning_clear()
    try:
        gpu.cnn_set_autotune(True)
        _, s1, e1 = kernel_timed_pass(model, xd, nl)       # tunes both conv shapes
        y2, s2, e2 = kernel_timed_pass(model, xd, nl)      # tuned
        gpu.cnn_set_autotune(False)
        assert len(gpu.cnn_tuning_export().splitlines()) == 2
    finally:
        gpu.cnn_set_autotune(False)
        gpu.cnn_tuning_clear()
    for i, layer in enumerate(net.layers):
        if layer.kind == "conv":
            first, tuned = s1[i].elapsed_time(e1[i]), s2[i].elapsed_time(e2[i])
            assert 0 < first < 3 * tuned + 0.05, (i, first, tuned)


def test_standalone_relu_layer_is_folded(gpu):
    """A RELU layer after conv / pool runs inside that layer; the result is the same
    as the oracle's separate ReLU."""
    net = wl.Net("relu_chain", (3, 16, 16), (
        wl.relu(),                       # first layer: standalone
        wl.conv(3, 8, 3, pad=1), wl.relu(),
        wl.pool("max", 2, 2), wl.relu(),
        wl.lrn(), wl.relu(),             # after LRN: standalone, in place
        wl.fc(8 * 8 * 8, 10), wl.relu(),
    ), weight_std=0.3, bias_std=0.1, input_dist="normal")
    x = wl.make_input(net, 4, 4)
    params = wl.make_params(net, 4)
    y = to_host(gpu.Network(net, params)(to_dev(x)))
    assert_gemm_close(y, oracle.net_fwd(net, x, params), 512, "relu chain")


def test_net_output_canary_and_workspace_reuse(gpu):
    net = wl.lenet
    model = gpu.Network(net, wl.make_params(net, 5))
    for batch in (16, 3, 16):
        x = wl.make_input(net, batch, 5)
        buf = torch.full((batch * 10 + 1024,), -777.0, device="cuda")
        model(to_dev(x), y=buf[: batch * 10].view(batch, 10))
        out = to_host(buf)
        assert np.all(out[batch * 10:] == -777.0)
        assert_gemm_close(out[: batch * 10].reshape(batch, 10),
                          oracle.net_fwd(net, x, wl.make_params(net, 5)), 500, f"lenet B{batch}")


@pytest.mark.parametrize("C,H,mode,k,s,p,relu,batch", [
    (96, 55, "max", 3, 2, 0, False, 3),    # AlexNet layers 2-3 shape
    (40, 27, "max", 3, 2, 1, True, 3),     # channel count not a multiple of 8, padding, ReLU
    (7, 13, "avg", 3, 2, 0, False, 3),
    (33, 9, "max", 2, 2, 0, False, 3),
    (5, 120, "max", 3, 2, 0, False, 3),
    # batches large enough for 16-channel workgroups
    (256, 27, "max", 3, 2, 0, False, 16),  # AlexNet layers 6-7 shape
    (72, 27, "max", 3, 2, 1, True, 64),    # 72 channels: last chunk of 16 ragged
    (72, 27, "avg", 3, 2, 1, False, 64),
])
def test_lrn_then_pool_matches_separate_layers(gpu, C, H, mode, k, s, p, relu, batch):
    """An LRN followed by pooling in a network gives values and indices equal,
    bit for bit, to those of the two single-layer calls."""
    print(f"lrn+pool C{C} H{H} {mode} k{k} s{s} p{p} relu{int(relu)} batch {batch}", flush=True)
    net = wl.Net("lrn_pool", (C, H, H), (wl.lrn(5, 1e-2, 0.75, 2.0),
                                        wl.pool(mode, k, s, p, relu=relu)),
                 weight_std=0.0, bias_std=0.0, input_dist="normal")
    x = wl.make_input(net, batch, 8) * 4
    model = gpu.Network(net, wl.make_params(net, 8), pool_index=(mode == "max"))
    xd = to_dev(x)
    y = to_host(model(xd))
    l = gpu.cnn_lrn_fwd(xd, 5, 1e-2, 0.75, 2.0)
    r = gpu.cnn_pool_fwd(l, mode, k, s, p, True, relu, with_index=(mode == "max"))
    if mode == "max":
        np.testing.assert_array_equal(y, to_host(r[0]))
        np.testing.assert_array_equal(to_host(model.indices[1]), to_host(r[1]))
    else:
        np.testing.assert_array_equal(y, to_host(r))
    ref = oracle.pool_fwd(oracle.lrn_fwd(x, 5, 1e-2, 0.75, 2.0), mode, (k, k), (s, s), (p, p), True, relu)
    np.testing.assert_allclose(y, ref, rtol=2e-5, atol=1e-6 * np.abs(x).max())


def test_nets_with_softmax(gpu):
    """LeNet with a softmax after its last FC (one row per image) and a small
    net with a softmax across the channels of a conv output, mid-network."""
    lenet_sm = wl.Net("lenet_softmax", wl.lenet.input_chw, wl.lenet.layers + (wl.softmax(),),
                      wl.lenet.weight_std, 1.0, input_dist="normal")
    mid = wl.Net("conv_softmax", (3, 16, 16), (
        wl.conv(3, 12, 3, pad=1, relu=True), wl.softmax(), wl.pool("max", 2, 2),
        wl.conv(12, 8, 3), wl.softmax(), wl.fc(8 * 6 * 6, 10), wl.softmax(),
    ), 0.3, 0.1, input_dist="normal")
    for net, batch in ((lenet_sm, 16), (mid, 5)):
        print(f"net {net.name} batch {batch}", flush=True)
        x = wl.make_input(net, batch, 9)
        params = wl.make_params(net, 9)
        y = to_host(gpu.Network(net, params)(to_dev(x)))
        ref = oracle.net_fwd(net, x, params)
        assert y.shape == ref.shape
        # a logit error e changes a probability by a factor exp(e): the FC
        # criterion on the logits becomes a relative one on the output
        np.testing.assert_allclose(y, ref, rtol=1e-4, atol=1e-30)
        np.testing.assert_allclose(y.astype(np.float64).sum(axis=1), 1.0, rtol=1e-5)


@pytest.mark.parametrize("mode", ["parallel", "graph"])
def test_alexnet_from_netfile(gpu, mode):
    """The shipped AlexNet NetFile, run in each execution mode, against the
    oracle on sampled images of a batch of 16."""
    import os
    print(f"alexnet netfile {mode}", flush=True)
    text = open(os.path.join(gpu.NETFILE_DIR, "alexnet.txt")).read().replace(
        "execution_mode parallel", f"execution_mode {mode}")
    nf = gpu.parse_netfile(text, weight_std=0.01, bias_std=0.01)
    assert nf.execution_mode == mode
    params = wl.make_params(nf.net, 10)
    x = wl.make_input(nf.net, 16, 10)
    xd = to_dev(x)
    try:
        model = gpu.Network.from_netfile(nf, params)   # the file asks for auto-tuning
        for _ in range(2):                              # graph mode: capture, then replay
            y = to_host(model(xd))
            assert_gemm_close(y[[0, 15]], oracle.net_fwd(nf.net, x[[0, 15]], params), 4096,
                              f"netfile {mode}")
    finally:
        gpu.cnn_set_autotune(False)


@pytest.mark.parametrize("batch", [1, 17, 70])
def test_fc_chain_relu_carried_into_next_layer(gpu, batch):
    """FC+ReLU layers that split their reduction leave the ReLU to the next FC
    layer, which applies it as it reads its input; half of the pre-activations
    are negative here, so a lost or doubled ReLU shows."""
    print(f"fc chain batch {batch}", flush=True)
    net = wl.Net("fc_chain", (8, 8, 8), (
        wl.fc(512, 300, relu=True), wl.fc(300, 200), wl.relu(), wl.fc(200, 10),
    ), 0.2, 0.2, input_dist="normal")
    x = wl.make_input(net, batch, 11)
    params = wl.make_params(net, 11)
    y = to_host(gpu.Network(net, params)(to_dev(x)))
    assert_gemm_close(y, oracle.net_fwd(net, x, params), 200, f"fc chain B{batch}")


@pytest.mark.parametrize("name,batch", [("alexnet", 1), ("alexnet", 2), ("lenet", 1),
                                        ("cifar_quick", 1), ("cifar_quick", 3)])
def test_small_batches(gpu, name, batch):
    """Small batches split the conv and FC reductions: their outputs start as
    the bias (one fill for the pass) and their ReLUs are applied by the next
    layer as it reads them (conv gathers, pooling, LRN, FC)."""
    run_layers(gpu, wl.NETS[name], batch, None, seed=12)


def test_workspace_size_does_not_depend_on_tuning(gpu):
    net = wl.alexnet
    params = wl.make_params(net, 13)
    x = to_dev(wl.make_input(net, 2, 13))
    gpu.cnn_tuning_clear()
    try:
        gpu.cnn_set_autotune(True)
        model = gpu.Network(net, params)
        before = model.workspace_bytes(2)
        y1 = to_host(model(x))            # tunes every conv shape of batch 2
        assert model.workspace_bytes(2) == before
        y2 = to_host(model(x))            # tuned configurations, maybe split
        assert_gemm_close(y2, y1, 4096, "tuned vs first pass")
    finally:
        gpu.cnn_set_autotune(False)
        gpu.cnn_tuning_clear()


def test_replicas_run_concurrently_on_two_streams(gpu):
    """Network.replica shares the device parameters but not the workspace:
    passes of the two on two streams, in flight together, each match the
    oracle on their own input (with indices for the max-pooling layers)."""
    net = wl.lenet
    params = wl.make_params(net, 14)
    model = gpu.Network(net, params, pool_index=True)
    rep = model.replica()
    assert rep.weights is model.weights
    xs = [wl.make_input(net, 16, 14), wl.make_input(net, 16, 15)]
    xd = [to_dev(x) for x in xs]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    ys = [None, None]
    torch.cuda.synchronize()
    for _ in range(3):
        for j, m in enumerate((model, rep)):
            with torch.cuda.stream(streams[j]):
                ys[j] = m(xd[j], stream=streams[j])
    torch.cuda.synchronize()
    for j, m in enumerate((model, rep)):
        ref, outs, ref_idx = oracle.net_fwd(net, xs[j], params, keep=True, pool_index=True)
        assert_gemm_close(to_host(ys[j]), ref, net.layers[-1].in_features, f"replica {j}")
        kred = None
        for i, layer in enumerate(net.layers):
            if layer.kind == "conv":
                kred = layer.in_channels * layer.kernel[0] * layer.kernel[1]
            if layer.kind == "pool" and layer.mode == "max":
                check_index_near_ties(layer, outs[i - 1], to_host(m.indices[i]), ref_idx[i],
                                      1e-4 * np.sqrt(kred), f"replica {j} layer {i}")


@pytest.mark.parametrize("batch", [1, 3, 16])
@pytest.mark.parametrize("pad", [(1, 1), (2, 1), (2, 2)])
@pytest.mark.parametrize("pool", [("max", 3, 2, 0), ("avg", 3, 1, 1)])
def test_padded_conv_after_lrn_pool(gpu, batch, pad, pool):
    """An LRN + pooling kernel followed by a padded convolution writes its
    output planes inside a zero border and the convolution runs unpadded on
    them.  Several bands and channel chunks per image, border widths that
    differ by axis, a ReLU folded into the pooling, and max-pool indices,
    which keep the plain layout."""
    mode, pk, ps, pp = pool
    print(f"lrn+pool {pool} -> conv pad {pad} batch {batch}", flush=True)
    k = (2 * pad[0] + 1, 2 * pad[1] + 1)
    P, Q = oracle.pool_out_shape(29, 23, pk, pk, ps, ps, pp, pp)
    net = wl.Net("lrn_pool_conv", (40, 29, 23), (
        wl.lrn(5, 1e-2, 0.75, 2.0), wl.pool(mode, pk, ps, pp), wl.relu(),
        wl.conv(40, 24, k, 1, pad, 2, relu=True),
        wl.fc(24 * P * Q, 10),
    ), 0.1, 0.1, input_dist="normal")
    x = wl.make_input(net, batch, 16) * 3
    params = wl.make_params(net, 16)
    model = gpu.Network(net, params, pool_index=(mode == "max"))
    _y, ref, ref_idx = oracle.net_fwd(net, x, params, keep=True, pool_index=True)
    y, outs, written = model.forward_dump(to_dev(x))
    torch.cuda.synchronize()
    g = [None if o is None else o.cpu().numpy() for o in outs]
    gi = [None if t is None else t.cpu().numpy() for t in model.indices]
    assert written == [True, True, False, True, True]    # the ReLU runs inside the pooling
    np.testing.assert_array_equal(to_host(y), g[-1])
    y2 = to_host(model(to_dev(x)))
    assert_gemm_close(y2, ref[-1], 24 * P * Q, f"{pool} pad {pad} B{batch}")
    compare_layers(net, params, x, g, written, ref, gi, ref_idx, f"{pool} pad {pad} B{batch}")


# Conv chains straight from conv to conv: pads of 1 and 2, unequal row and
# column pads, a strided and a grouped producer, a ReLU folded into the
# producer, a 1x1 conv in between.
CONV_CHAIN_NET = wl.Net(
    name="conv_chain",
    input_chw=(6, 15, 17),
    layers=(
        wl.conv(6, 16, 3, 2, 1, relu=True),
        wl.conv(16, 24, 3, 1, 1, groups=2),
        wl.relu(),
        wl.conv(24, 20, (3, 5), 1, (1, 2)),
        wl.conv(20, 8, 1),
        wl.conv(8, 12, 3, 1, 1, relu=True),
        wl.conv(12, 12, (1, 3), 1, (0, 1)),
        wl.fc(12 * 8 * 9, 10),
    ),
    weight_std=0.1, bias_std=0.05,
)


@pytest.mark.parametrize("batch", [1, 4, 16])
def test_conv_chain(gpu, batch):
    """Batch 1 splits every conv's reduction (outputs prefilled with the bias,
    ReLUs left to the next conv); 4 and 16 do not split the larger layers."""
    print(f"net conv_chain batch {batch}", flush=True)
    x = wl.make_input(CONV_CHAIN_NET, batch, 21)
    dump_and_compare(gpu, CONV_CHAIN_NET, wl.make_params(CONV_CHAIN_NET, 21), x)
