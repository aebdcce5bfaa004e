import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workload (minutes of host generation)")


@pytest.fixture(scope="session")
def gpu():
    """The HIP library bound to cuda:0; GPU tests fail loudly without it."""
    import torch
    assert torch.cuda.is_available(), "GPU test run without a visible GPU"
    from paper_2606_29207_amd import kf
    kf.load()
    return kf
