import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workloads (minutes of host time)")


@pytest.fixture(scope="session")
def gpu_lib():
    """The HIP library through its Python binding; a GPU test fails loudly
    (not skips) when the library or the device is missing."""
    import torch
    from paper_2606_07665_amd import binding
    assert torch.cuda.is_available(), "GPU test run without a visible GPU"
    binding.load()
    return binding
