import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def oracle_lib():
    """Path of the built oracle library (built once if absent)."""
    import oracle
    from oracle import build
    path = os.environ.get("SL_ORACLE_LIBRARY") or build.LIBRARY
    oracle.load(path)
    return path
