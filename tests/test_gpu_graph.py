"""A captured HIP graph of cnn_net_fwd replays correctly (GPU).

Captured graphs of library calls have replayed wrong results on some
configurations when they held memset nodes; the network executor records
only kernels.  Each replay is checked against the eager result, with eager
work and synchronisations between the replays.
"""
import numpy as np
import pytest
import torch

from conftest import to_dev
from paper_1511_07376_amd import workloads as wl
from parity import assert_gemm_close

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,batch", [("lenet", 16), ("cifar_quick", 32), ("alexnet", 16)])
def test_graph_replays_match_eager(gpu, name, batch):
    print(f"graph replay {name} batch {batch}", flush=True)
    net = wl.NETS[name]
    model = gpu.Network(net, wl.make_params(net, 7))
    x = to_dev(wl.make_input(net, batch, 7))
    y_eager = model(x).clone()
    torch.cuda.synchronize()
    y = torch.empty_like(y_eager)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        model(x, y=y)
    kred = net.layers[-1].in_features
    for i in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert_gemm_close(y.cpu().numpy(), y_eager.cpu().numpy(), kred, f"replay {i}")
        other = model(x)            # eager work between replays
        torch.cuda.synchronize()
        assert np.isfinite(other.cpu().numpy()).all()


@pytest.mark.parametrize("name,batch", [("lenet", 16), ("cifar_quick", 32), ("alexnet", 16), ("lenet", 1)])
def test_library_graph_mode_replays(gpu, name, batch):
    """execution_mode "graph": the library captures the network itself
    (cnn_net_graph_create) and each later call is one graph launch.  New
    input data copied into the same buffer between replays, eager work in
    between; every replay matches the eager network on that data."""
    print(f"library graph mode {name} batch {batch}", flush=True)
    net = wl.NETS[name]
    params = wl.make_params(net, 8)
    eager = gpu.Network(net, params)
    graphed = gpu.Network(net, params, execution_mode="graph")
    x = to_dev(wl.make_input(net, batch, 8))
    kred = net.layers[-1].in_features
    y0 = graphed(x)                      # eager pass + capture
    assert_gemm_close(y0.cpu().numpy(), eager(x).cpu().numpy(), kred, "first call")
    for i in range(3):
        x.copy_(to_dev(wl.make_input(net, batch, 100 + i)))
        y = graphed(x)                   # replay
        assert y.data_ptr() == y0.data_ptr() and len(graphed._graphs) == 1
        torch.cuda.synchronize()
        ref = eager(x)
        torch.cuda.synchronize()
        assert_gemm_close(y.cpu().numpy(), ref.cpu().numpy(), kred, f"replay {i}")
    # another batch size: a second workspace, old graphs dropped
    x2 = to_dev(wl.make_input(net, batch + 1, 9))
    assert_gemm_close(graphed(x2).cpu().numpy(), eager(x2).cpu().numpy(), kred, "new batch")
    assert_gemm_close(graphed(x2).cpu().numpy(), eager(x2).cpu().numpy(), kred, "new batch replay")
    graphed.close()


def test_graph_create_rejects_and_handles_empty_batch(gpu):
    import ctypes
    net = wl.lenet
    model = gpu.Network(net, wl.make_params(net, 1))
    g = ctypes.c_void_p()
    # workspace too small: nothing captured, no handle
    rc = gpu.lib.cnn_net_graph_create(model.descs, len(model.descs), 0x1000, 2, 1, 28, 28, 0x1000,
                                      0x1000, 16, ctypes.byref(g))
    assert rc == gpu.CNN_ERR_WORKSPACE and not g.value
    assert gpu.lib.cnn_net_graph_launch(None, None) == gpu.CNN_ERR_INVALID
    assert gpu.lib.cnn_net_graph_destroy(None) == 0
    rc = gpu.lib.cnn_net_graph_create(model.descs, len(model.descs), None, 0, 1, 28, 28, None, None, 0,
                                      ctypes.byref(g))
    assert rc == 0 and g.value
    assert gpu.lib.cnn_net_graph_launch(g, None) == 0
    assert gpu.lib.cnn_net_graph_destroy(g) == 0
