import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test")


def pytest_terminal_summary(terminalreporter):
    """Loss-change precision, tie band and decision flips of every GPU parity
    run of the session (shown in -q runs too)."""
    try:
        from parity_util import REPORTS
    except Exception:
        return
    used = [r for r in REPORTS if r.n]
    if used:
        terminalreporter.write_sep("-", "parity: loss changes against the oracle")
        for r in used:
            terminalreporter.write_line(str(r))
