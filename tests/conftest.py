import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (run through the C ABI on cuda:0)")
    config.addinivalue_line("markers", "slow: exhaustive CPU sweeps (still part of the CPU suite)")


@pytest.fixture(scope="session")
def oracle():
    import oracle as o
    o.lib()
    return o
