import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long CPU test")


def pytest_collection_modifyitems(config, items):
    # Run GPU tests in file order but after CPU tests of the same file.
    pass


@pytest.fixture(scope="session")
def gpu():
    """A CUDA/HIP device; GPU tests fail loudly when the library is missing."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this container")
    return torch.device("cuda:0")
