import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def lib():
    """The built C-ABI library (built once if missing)."""
    from paper_1512_02673_amd import build as _build
    if not os.path.exists(_build.LIB_PATH):
        _build.build()
    from paper_1512_02673_amd import binding
    return binding
