import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built libkvx.so")


@pytest.fixture(scope="session")
def gpu_kvx():
    """The HIP binding on cuda:0; fails loudly when the library is missing."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("gpu test selected but no GPU is visible")
    from paper_2608_03893_amd import kvx
    kvx.load()
    return kvx
