import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs a gfx950 GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU-side oracle runs")


@pytest.fixture(scope="session")
def gpu_lib():
    """The built HIP library with a visible GPU; GPU tests fail loudly without it."""
    import torch
    from paper_2505_17074_amd import binding
    if not torch.cuda.is_available():
        pytest.fail("GPU test selected but no GPU is visible")
    lib = binding.load()
    return lib
