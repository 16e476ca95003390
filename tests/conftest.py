import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running test")


def _stale(lib, srcs):
    if not os.path.exists(lib):
        return True
    t = os.path.getmtime(lib)
    return any(os.path.getmtime(s) > t for s in srcs)


@pytest.fixture(scope="session", autouse=True)
def _oracle_built():
    """The oracle is plain C built with gcc; (re)build it when missing or stale
    so the CPU tests always run the committed source."""
    from oracle import build as ob
    if _stale(ob.LIB, [os.path.join(ob.HERE, "zo_oracle.c")]):
        ob.build()
    yield
