import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built libfem.so")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def gpu_available():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def fem():
    """The HIP binding; a GPU test fails loudly if the library is missing."""
    if not gpu_available():
        pytest.skip("no GPU visible")
    from paper_2602_07160_amd import binding
    binding.load()  # raises if libfem.so is absent
    return binding
