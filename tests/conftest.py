import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an AMD GPU (MI355X); runs the HIP kernels")


@pytest.fixture(scope="session")
def orc():
    """The CPU oracle, built from source if its library is absent."""
    import oracle
    oracle.lib()
    return oracle


@pytest.fixture(scope="session")
def gpu():
    """torch with a visible GPU and the built codec library; GPU tests fail (not skip) when
    the library is missing, so a GPU run can never pass without the native path."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2603_27467_amd as tvq
    tvq.load_library()
    return torch
