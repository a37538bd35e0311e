import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running full-size case")


@pytest.fixture(scope="session")
def gpu_lib():
    """The HIP-backed binding; GPU tests fail loudly if it cannot load."""
    import torch

    # device_count() does not initialise the GPU (is_available() does), so that
    # inputs generated after this fixture may still use worker processes
    if torch.cuda.device_count() < 1:
        pytest.fail("GPU test selected but no GPU is visible")
    from paper_2608_10519_amd import sparstar

    sparstar.load()  # raises if the library is missing
    return sparstar
