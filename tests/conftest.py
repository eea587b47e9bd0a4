import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running case")


def pytest_terminal_summary(terminalreporter):
    from tests.util import OUTPUT_TALLY as t
    if t["calls"]:
        terminalreporter.write_line(
            f"output comparisons: {t['calls']} calls, {t['elements']} O elements, {t['over']} beyond 1e-2 "
            f"(worst {t['worst']:.4f})")
