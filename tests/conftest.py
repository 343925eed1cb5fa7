import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an AMD GPU (MI355X) and the built liblsgd.so")


@pytest.fixture(scope="session", autouse=True)
def _oracle_built():
    """The oracle library is test infrastructure: build it if it is missing."""
    from oracle import build as oracle_build
    if not os.path.exists(oracle_build.LIB):
        oracle_build.build()
    yield
