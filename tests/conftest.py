import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU oracle case")
    config.addinivalue_line("markers", "fullsize: GPU parity at a workload's full size (minutes of host work)")


def pytest_collection_modifyitems(config, items):
    # GPU tests run in file order, but the allocation-free entry point's test
    # (if present) is kept last so a failure there cannot hide the others.
    items.sort(key=lambda it: 1 if "test_zz_" in it.nodeid else 0)


def ensure_built():
    """Build the library if nothing is built, or if what is built does not
    match the sources in this tree (bc_build_id against the source hash)."""
    import paper_2608_28670_amd as bc
    if not bc.is_current():
        from paper_2608_28670_amd import build
        print(f"libbarycache.so is missing or stale (build id {bc.built_id()}); rebuilding", file=sys.stderr)
        build.build()


@pytest.fixture(scope="session")
def bclib():
    ensure_built()
    import paper_2608_28670_amd as bc
    bc.lib()
    return bc
