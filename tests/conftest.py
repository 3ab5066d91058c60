import os
import sys

import numpy as np
import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if REPO not in sys.path:
    sys.path.insert(0, REPO)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU; runs the HIP kernels")


def has_gpu_node() -> bool:
    """True if this machine exposes a ROCm GPU device node (checked without
    initializing HIP)."""
    return os.path.exists("/dev/kfd")


@pytest.fixture(scope="session")
def rng():
    return np.random.default_rng(12345)
