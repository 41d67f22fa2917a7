import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Tolerance margins (max err/bound per checked tensor) of the run."""
    try:
        from _common import MARGINS
    except ImportError:
        return
    if not MARGINS:
        return
    terminalreporter.write_sep("-", "tolerance margins (max err / bound; < 1 passes)")
    for test, name, ratio in MARGINS:
        terminalreporter.write_line(f"{ratio:8.3f}  {name:40s} {test}")
