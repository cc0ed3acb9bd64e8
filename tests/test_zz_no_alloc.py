"""cnn_net_fwd_noalloc (GPU): the network pass on the library's static
device scratch, called through the C ABI, against cnn_net_fwd (the same
network with a caller workspace) and the oracle.  Two calls in a row on
each network, the second with a smaller batch, so that the second reuses a
scratch that still holds the first's intermediates; an input that needs more
than the scratch is refused before anything is enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from conftest import to_dev, to_host
from paper_1511_07376_amd import workloads as wl
from parity import assert_gemm_close

pytestmark = pytest.mark.gpu


def _noalloc(gpu, model, x, y):
    N, C, H, W = x.shape
    rc = gpu.lib.cnn_net_fwd_noalloc(model.descs, len(model.descs), x.data_ptr(), N, C, H, W, y.data_ptr(),
                                     torch.cuda.current_stream().cuda_stream)
    assert rc == gpu.CNN_OK, gpu.cnn_last_error()
    return y


@pytest.mark.parametrize("name,batches,sample", [
    ("cifar_quick", (32, 8), None),
    ("lenet", (256, 16), [0, 100, 255]),
    ("alexnet", (64, 16), [0, 63]),
])
def test_noalloc_matches_workspace_entry_point(gpu, name, batches, sample):
    net = wl.NETS[name]
    params = wl.make_params(net, 30)
    model = gpu.Network(net, params)
    kred = [l for l in net.layers if l.kind == "fc"][-1].in_features
    for call, batch in enumerate(batches):
        print(f"noalloc {name} call {call} batch {batch}", flush=True)
        assert model.workspace_bytes(batch) <= gpu.CNN_NOALLOC_SCRATCH_BYTES
        x = wl.make_input(net, batch, 31 + call)
        xd = to_dev(x)
        y = torch.full(model.out_shape(batch), float("nan"), device="cuda")
        _noalloc(gpu, model, xd, y)
        got = to_host(y)
        ref_ws = to_host(model(xd))          # cnn_net_fwd with a caller workspace
        assert_gemm_close(got, ref_ws, kred, f"{name} B{batch} vs cnn_net_fwd")
        rows = list(range(batch)) if sample is None else [r for r in sample if r < batch]
        assert_gemm_close(got[rows], oracle.net_fwd(net, x[rows], params), kred, f"{name} B{batch} vs oracle")


def test_noalloc_refuses_inputs_beyond_the_scratch(gpu):
    net = wl.alexnet
    model = gpu.Network(net, wl.make_params(net, 32))
    batch = 128
    assert model.workspace_bytes(batch) > gpu.CNN_NOALLOC_SCRATCH_BYTES
    x = torch.zeros((batch,) + net.input_chw, device="cuda")
    y = torch.full(model.out_shape(batch), -5.0, device="cuda")
    rc = gpu.lib.cnn_net_fwd_noalloc(model.descs, len(model.descs), x.data_ptr(), batch, *net.input_chw,
                                     y.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert rc == gpu.CNN_ERR_WORKSPACE
    assert "static scratch" in gpu.cnn_last_error()
    assert bool(torch.all(y == -5.0))


def test_noalloc_does_not_tune(gpu):
    """With auto-tuning on, the no-allocation pass still runs (the heuristic's
    configurations, no timing runs) and records nothing."""
    net = wl.cifar_quick
    params = wl.make_params(net, 33)
    model = gpu.Network(net, params)
    x = wl.make_input(net, 4, 33)
    gpu.cnn_tuning_clear()
    try:
        gpu.cnn_set_autotune(True)
        y = model.forward_noalloc(to_dev(x))
        torch.cuda.synchronize()
        assert gpu.cnn_tuning_export() == ""
    finally:
        gpu.cnn_set_autotune(False)
        gpu.cnn_tuning_clear()
    assert_gemm_close(to_host(y), oracle.net_fwd(net, x, params), 64, "noalloc with auto-tuning on")
