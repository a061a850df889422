import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) and the built HIP library")


@pytest.fixture(scope="session")
def tg():
    """The HIP library binding; on a GPU run a missing build is an error."""
    import paper_2608_26112_amd as tg_mod
    tg_mod.load()  # raises if libtreegraft.so is not built
    return tg_mod
