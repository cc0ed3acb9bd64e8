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
