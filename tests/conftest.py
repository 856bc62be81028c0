import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP kernels)")


@pytest.fixture(scope="session", autouse=True)
def _built_libraries():
    """Build the oracle and libleap only when nothing is built yet."""
    import oracle
    if not os.path.exists(oracle._LIB_PATH):
        oracle.build()
    from paper_2608_01804_amd import _build
    if not os.path.exists(_build.LIB_PATH):
        _build.build()
    yield
