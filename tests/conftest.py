import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test (full-size oracle runs)")


def pytest_terminal_summary(terminalreporter):
    """Print every parity check's counts (also when the run is quiet)."""
    helpers = sys.modules.get("tests.helpers")
    lines = getattr(helpers, "PARITY_LINES", None) if helpers else None
    if lines:
        terminalreporter.write_sep("-", "parity counts")
        for line in lines:
            terminalreporter.write_line(line)
