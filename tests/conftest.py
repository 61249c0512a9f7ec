import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the HIP library)")
    config.addinivalue_line("markers", "slow: full-size workload parity (minutes)")


def pytest_terminal_summary(terminalreporter):
    """Print the measured parity figures the GPU tests recorded (harness.REPORT)."""
    h = sys.modules.get("harness")
    lines = getattr(h, "REPORT", None) if h is not None else None
    if lines:
        terminalreporter.write_sep("-", "parity report (measured errors, counts)")
        for line in lines:
            terminalreporter.write_line(line)
