import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU oracle case")


def pytest_collection_modifyitems(config, items):
    # GPU tests run in file order, but the allocation-free entry point's test
    # (if present) is kept last so a failure there cannot hide the others.
    items.sort(key=lambda it: 1 if "test_zz_" in it.nodeid else 0)


def ensure_built():
    """Build the library if nothing is built yet (the driver builds first)."""
    from paper_2608_28670_amd import LIB_PATH
    if not os.path.exists(LIB_PATH):
        from paper_2608_28670_amd import build
        build.build()


@pytest.fixture(scope="session")
def bclib():
    ensure_built()
    import paper_2608_28670_amd as bc
    bc.lib()
    return bc
