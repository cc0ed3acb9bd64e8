"""The C ABI used from a C program with the HIP runtime and no Python or
torch in between (tests/c_abi/cifar_quick_c.c): CIFAR-10 quick described
with cnn_layer_desc, run by cnn_net_fwd, checked against the oracle's layers
chained in C.  The program is built with the library (`build()`); the GPU
test runs it as a child process."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "c_abi"))
import build_c_abi as c_build  # noqa: E402

PROGRAM = c_build.PROGRAM


def test_c_program_builds():
    """Compiles against include/cnn.h and oracle/oracle.h (CPU)."""
    pytest.importorskip("paper_1511_07376_amd.cnn", reason="libcnn.so not built")
    assert os.path.exists(c_build.build())


@pytest.mark.gpu
def test_c_program_matches_oracle(gpu):
    assert os.path.exists(PROGRAM), "build it first: python __graft_entry__.py"
    print("cifar_quick_c", flush=True)
    r = subprocess.run([PROGRAM], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert "max abs err" in r.stdout
