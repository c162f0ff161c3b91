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


def pytest_terminal_summary(terminalreporter):
    """The elementwise size of the fp32 errors, beside the normwise verdicts the tests apply."""
    from tests.helpers import FP32_ELEMENTWISE

    if not FP32_ELEMENTWISE:
        return
    worst = sorted(FP32_ELEMENTWISE, key=lambda t: -t[1])
    tr = terminalreporter
    tr.write_sep("-", "fp32 outputs, elementwise")
    tr.write_line(f"{len(FP32_ELEMENTWISE)} fp32 comparisons; largest |x-r| / (1e-5|r| + 1e-5 rms(r)): "
                  f"{worst[0][1]:.3g} ({worst[0][0]}); largest |x-r|/|r| where |r| >= rms(r): "
                  f"{max(t[2] for t in FP32_ELEMENTWISE):.3g}")
    over = [t for t in worst if t[1] > 1.0]
    tr.write_line(f"{len(over)} of them exceed the elementwise reading of the bar; worst ten:")
    for name, ratio, rel in worst[:10]:
        tr.write_line(f"  {name}: ratio {ratio:.3g}, max rel {rel:.3g}")
