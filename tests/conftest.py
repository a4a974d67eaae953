import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session")
def nnlib():
    """libnnconv, built in-tree first if no build is present."""
    from paper_2102_06725_amd import nnconv
    if not os.path.exists(nnconv.LIB_PATH):
        from paper_2102_06725_amd import build
        build.build()
    return nnconv.load()


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle.oracle as orc
    orc.build(force=False)
    return orc.load()
