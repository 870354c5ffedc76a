import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="module", autouse=True)
def _stated_bar_over_the_module(request):
    """Sum the stored entries that differ from the oracle over every fused-step
    comparison of a module, and hold the sum to the 0.01 % bar at its end."""
    if "gpu" not in request.module.__name__:
        yield
        return
    from tests import _parity
    _parity.LEDGER.update(entries=0, differ=0, tests=[])
    yield
    _parity.check_ledger(request.module.__name__)


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle.lib()
    return oracle
