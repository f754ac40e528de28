import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size case, several seconds or more")


@pytest.fixture(scope="session", autouse=True)
def _library_built():
    """Build librpd.so once if it is missing (tests load what is built)."""
    lib = os.path.join(ROOT, "paper_2609_36452_amd", "librpd.so")
    if not os.path.exists(lib):
        from paper_2609_36452_amd.build import build
        build()
    yield
