import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def gt():
    """The HIP library binding; the test fails (does not skip) when it cannot load on a GPU run."""
    import paper_2407_14106_amd as pkg

    return pkg.load()
