import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture
def rng():
    return np.random.default_rng(12345)


def pytest_terminal_summary(terminalreporter):
    # Whole-tensor parity figures of the full-size GPU runs (max and mean
    # scaled error, literal max-abs and mean-abs error, norm-wise error).
    parity = sys.modules.get("parity")
    lines = getattr(parity, "WHOLE_TENSOR_REPORT", None) if parity else None
    if lines:
        terminalreporter.section("whole-tensor parity against the oracle")
        for line in lines:
            terminalreporter.write_line(line)
