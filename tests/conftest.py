import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size oracle work (tens of seconds)")


@pytest.fixture(scope="session")
def gpu():
    """Skip unless a GPU and the HIP library are both present; the product
    path itself never falls back to anything when they are missing."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2512_02901_amd import binding
    binding.load()  # raises if the library is missing
    return torch.device("cuda:0")
