import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running case (full-size workload)")


@pytest.fixture(scope="session")
def gpu_lib():
    """The HIP library through its Python binding; a GPU test that cannot get
    it fails (it never falls back to anything else)."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("gpu test collected on a machine without a GPU")
    from paper_1903_05133_amd import native
    return native.lib()
