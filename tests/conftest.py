import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X and the HIP library")
    config.addinivalue_line("markers", "slow: larger CPU cases")


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle._L()
    return oracle


def pytest_terminal_summary(terminalreporter):
    """Whether each end-to-end label comparison ran under the separation
    guard (agreement) or not (k-means of the GPU's own v)."""
    helpers = sys.modules.get("gpu_helpers")
    lines = getattr(helpers, "LABEL_GUARD", None)
    if lines:
        terminalreporter.section("label parity guard")
        for line in lines:
            terminalreporter.write_line(line)
