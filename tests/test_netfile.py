"""NetFile parsing (cnn_netfile_parse; host only, no GPU).

The paper configures its engine with a text file listing the layers and
three parameters, allocated_ram, execution_mode and auto_tuning (Sec. 3.2);
its syntax is in a figure that is not reproduced, so the syntax is this
library's own (documented in cnn.h).  The NetFiles shipped for the three
networks of the paper's layer-setup table must describe exactly the layer
lists the tests and the benchmark use.
"""
import ctypes
import os

import numpy as np
import pytest

from paper_1511_07376_amd import cnn
from paper_1511_07376_amd import workloads as wl


def _same_layers(a, b):
    """Layer lists equal, LRN constants compared at float32 (the descriptor's
    precision)."""
    assert len(a) == len(b)
    for x, y in zip(a, b):
        if x.kind == "lrn":
            assert y.kind == "lrn" and x.size == y.size
            for f in ("alpha", "beta", "k"):
                assert np.float32(getattr(x, f)) == np.float32(getattr(y, f))
        else:
            assert x == y


@pytest.mark.parametrize("name", ["lenet", "cifar_quick", "alexnet"])
def test_shipped_netfiles_describe_the_paper_nets(name):
    nf = cnn.load_netfile(os.path.join(cnn.NETFILE_DIR, f"{name}.txt"))
    ref = wl.NETS[name]
    assert nf.net.input_chw == ref.input_chw
    _same_layers(nf.net.layers, ref.layers)
    assert nf.execution_mode == "parallel"
    assert nf.auto_tuning == (name == "alexnet")


def test_syntax_defaults_and_parameters():
    text = """
    # a comment line
    input: 3 16 12          # colon form, trailing comment
    execution_mode: graph
    auto_tuning 1
    allocated_ram 512

    conv out=8 kernel=3x5 pad=1x2 relu
    lrn
    pool avg kernel=3 stride=2 ceil=0
    relu
    conv out=6 kernel=1 groups=2
    fc out=7
    softmax
    """
    nf = cnn.parse_netfile(text)
    assert nf.execution_mode == "graph" and nf.auto_tuning and nf.allocated_ram_mib == 512
    L = nf.net.layers
    assert nf.net.input_chw == (3, 16, 12)
    assert L[0] == wl.conv(3, 8, (3, 5), 1, (1, 2), 1, True)
    assert L[1].kind == "lrn" and L[1].size == 5 and np.float32(L[1].alpha) == np.float32(1e-4)
    assert L[1].beta == 0.75 and L[1].k == 1.0
    assert L[2] == wl.pool("avg", 3, 2, 0, ceil=False)
    assert L[3] == wl.relu()
    # shapes follow the library's rules: 16x12 conv -> 16x12, avg pool floor -> 7x5
    assert L[4] == wl.conv(8, 6, 1, 1, 0, 2)
    assert L[5] == wl.fc(6 * 7 * 5, 7)
    assert L[6] == wl.softmax()


def test_count_only_call_and_input_override():
    n = ctypes.c_int()
    cfg = cnn.cnn_netfile_config()
    text = b"conv out=4 kernel=3\nrelu\nfc out=2\n"
    assert cnn.lib.cnn_netfile_parse(text, None, 0, ctypes.byref(n), ctypes.byref(cfg)) == 0
    assert n.value == 3 and cfg.in_channels == 0 and cfg.execution_mode == cnn.CNN_EXEC_PARALLEL
    descs = (cnn.cnn_layer_desc * 2)()
    assert cnn.lib.cnn_netfile_parse(text, descs, 2, ctypes.byref(n), ctypes.byref(cfg)) == cnn.CNN_ERR_INVALID
    assert "line 3" in cnn.cnn_last_error()
    with pytest.raises(ValueError):
        cnn.parse_netfile(text.decode())          # no input shape
    nf = cnn.parse_netfile(text.decode(), input_chw=(2, 5, 5))
    assert nf.net.layers[2] == wl.fc(4 * 3 * 3, 2)


@pytest.mark.parametrize("text,line,status,words", [
    ("conv out=4 kernel=3\nbogus 3\n", 2, cnn.CNN_ERR_INVALID, "unknown statement"),
    ("conv out=4 kernel=3 colour=red\n", 1, cnn.CNN_ERR_INVALID, "unknown option"),
    ("conv out=4 kernel=3 out=5\n", 1, cnn.CNN_ERR_INVALID, "twice"),
    ("\n\nconv out=-4 kernel=3\n", 3, cnn.CNN_ERR_INVALID, "bad value"),
    ("conv out=4 kernel=3x\n", 1, cnn.CNN_ERR_INVALID, "bad value"),
    ("conv out=4 kernel=0\n", 1, cnn.CNN_ERR_INVALID, "bad value"),
    ("conv out=4\n", 1, cnn.CNN_ERR_INVALID, "kernel="),
    ("fc relu\n", 1, cnn.CNN_ERR_INVALID, "out="),
    ("pool kernel=2\n", 1, cnn.CNN_ERR_INVALID, "mode"),
    ("pool max stride=2\n", 1, cnn.CNN_ERR_INVALID, "kernel="),
    ("pool max kernel=2 ceil=2\n", 1, cnn.CNN_ERR_INVALID, "bad value"),
    ("lrn alpha=abc\n", 1, cnn.CNN_ERR_INVALID, "bad value"),
    ("relu now\n", 1, cnn.CNN_ERR_INVALID, "no options"),
    ("conv out=4 kernel=3 relu=1\n", 1, cnn.CNN_ERR_INVALID, "no value"),
    ("conv out=4 kernel=3 stride\n", 1, cnn.CNN_ERR_INVALID, "needs a value"),
    ("input 3 32\n", 1, cnn.CNN_ERR_INVALID, "input"),
    ("execution_mode sequential\n", 1, cnn.CNN_ERR_UNSUPPORTED, "GPU"),
    ("execution_mode fast\n", 1, cnn.CNN_ERR_INVALID, "execution_mode"),
    ("auto_tuning maybe\n", 1, cnn.CNN_ERR_INVALID, "auto_tuning"),
    ("allocated_ram -1\n", 1, cnn.CNN_ERR_INVALID, "allocated_ram"),
])
def test_errors_name_the_line(text, line, status, words):
    n = ctypes.c_int()
    cfg = cnn.cnn_netfile_config()
    rc = cnn.lib.cnn_netfile_parse(text.encode(), None, 0, ctypes.byref(n), ctypes.byref(cfg))
    assert rc == status
    msg = cnn.cnn_last_error()
    assert msg.startswith(f"netfile line {line}:") and words in msg, msg


def test_layer_chain_errors_surface_on_conversion():
    """A declared in= that disagrees with the chain is caught by the shape rules."""
    with pytest.raises(cnn.CnnError, match="input channels"):
        cnn.parse_netfile("input 3 8 8\nconv out=4 kernel=3 in=5\n")
    with pytest.raises(cnn.CnnError, match="expects 10 inputs"):
        cnn.parse_netfile("input 3 8 8\nfc out=4 in=10\n")


def test_null_arguments():
    n = ctypes.c_int()
    cfg = cnn.cnn_netfile_config()
    assert cnn.lib.cnn_netfile_parse(None, None, 0, ctypes.byref(n), ctypes.byref(cfg)) == cnn.CNN_ERR_INVALID
    assert cnn.lib.cnn_netfile_parse(b"relu\n", None, 0, None, ctypes.byref(cfg)) == cnn.CNN_ERR_INVALID
    assert cnn.lib.cnn_netfile_parse(b"", None, 0, ctypes.byref(n), ctypes.byref(cfg)) == 0
    assert n.value == 0
