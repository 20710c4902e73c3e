import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs a real MI355X (runs through the C-ABI library)")
    config.addinivalue_line("markers", "slow: large CPU oracle case")


@pytest.fixture(scope="session", autouse=True)
def _oracle_built():
    """The oracle's C core is test infrastructure: build it once per session if absent."""
    from oracle import build as obuild
    lib = os.path.join(ROOT, "oracle", "liboracle.so")
    src = os.path.join(ROOT, "oracle", "ckks_oracle.c")
    if not os.path.exists(lib) or os.path.getmtime(lib) < os.path.getmtime(src):
        obuild.build()
    yield
