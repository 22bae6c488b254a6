import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def gpu():
    """The HIP library bound to cuda:0; fails (never skips) when the GPU or library is missing."""
    import torch
    assert torch.cuda.is_available(), "GPU test run without a visible GPU"
    import paper_2609_34325_amd as dora
    dora.load_library()
    return dora
