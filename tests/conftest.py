import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


import pytest  # noqa: E402


@pytest.fixture(scope="session")
def gpu():
    """The libcnn binding on a GPU.  Skips where there is no GPU; where there is
    one, a missing library is an error (the HIP path never falls back)."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this environment")
    from paper_1511_07376_amd import cnn
    return cnn


def to_dev(a):
    import torch
    return torch.from_numpy(a).cuda()


def to_host(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()
