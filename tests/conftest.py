import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) and the built HIP library")


def gpu_available():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def gpu():
    """Skip when no GPU is visible; otherwise hand back the binding.

    On a machine with a GPU the HIP library must load: a missing build is an
    error, never a silent skip or a fallback.
    """
    if not gpu_available():
        pytest.skip("no GPU visible")
    import paper_2505_08098_amd as f3s
    f3s.load_library()  # raises if libf3s.so is missing or unloadable
    return f3s


@pytest.fixture(scope="session")
def oracle():
    import oracle as orc
    orc.lib()
    return orc
