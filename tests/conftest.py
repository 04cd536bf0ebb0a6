import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def orc():
    from oracle import oracle
    return oracle.default()


@pytest.fixture(scope="session", autouse=True)
def built_library_matches_sources():
    """Every session that finds libheal.so checks that it was built from the
    sources in this tree, so that a stale binary cannot pass for the code."""
    from paper_2606_21023_amd import build as hbuild
    if os.path.exists(hbuild.LIBRARY):
        import paper_2606_21023_amd as heal
        heal.check_build()
    yield
