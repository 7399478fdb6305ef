import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


@pytest.fixture(scope="session")
def orc():
    from oracle import oracle
    oracle.lib()
    # all host cores (at most 16 threads): the
    # layer loops split output rows into bands, results are unchanged
    oracle.set_threads(max(1, min(16, os.cpu_count() or 1)))
    return oracle
