import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def gpu_lib():
    """The product binding, with its HIP library loaded; GPU tests only."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2604_08075_amd import binding
    return binding


@pytest.fixture(scope="session")
def host_lib():
    """The product binding for host-only calls (builds libdpool.so if nothing is built yet)."""
    from paper_2604_08075_amd import binding
    import os
    if not os.path.exists(binding.LIB_PATH):
        from paper_2604_08075_amd import build
        build.build()
    binding.lib()
    return binding
