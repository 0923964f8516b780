import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workload checks (minutes of oracle time)")


@pytest.fixture(scope="session")
def gpu_lib():
    """The loaded HIP binding; tests marked gpu fail loudly if it or the GPU is missing."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test collected on a host without a GPU")
    from paper_2606_20005_amd import streamkl
    return streamkl
