import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def _gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def gpu():
    """The HIP library bound to cuda:0; GPU tests fail (not skip) when the
    library is missing on a machine that has a GPU."""
    if not _gpu_available():
        pytest.skip("no GPU visible")
    import paper_2608_04048_amd as rrq
    rrq.load_library()
    return rrq
