import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running GPU check at full benchmark sizes")


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def ffmlp():
    """The GPU package with its library loaded; built here only if absent."""
    import paper_2403_17607_amd as pkg
    if not os.path.exists(pkg.LIB_PATH):
        from paper_2403_17607_amd import build
        build.build()
    pkg.lib()
    return pkg


@pytest.fixture(scope="session")
def gpu(ffmlp):
    """A GPU test that runs without a GPU is an error, not a silent pass."""
    if not gpu_available():
        pytest.fail("this test needs a GPU (run with -m 'not gpu' on a CPU host)")
    import torch
    return torch.device("cuda:0")
