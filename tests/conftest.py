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
    """Worst relative error of the importance scores per test (tests/parity.py
    records one entry per comparison)."""
    try:
        from parity import SCORE_RECORD
    except ImportError:
        return
    if not SCORE_RECORD:
        return
    worst = {}
    for test, where, rel, judged, floored in SCORE_RECORD:
        w = worst.setdefault(test, [0.0, 0, 0, 0])
        w[0] = max(w[0], rel)
        w[1] += judged
        w[2] += floored
        w[3] += 1
    terminalreporter.write_line("importance parity: worst relative error per test "
                                "(tokens judged relatively / under the floor, comparisons)")
    for test, (rel, judged, floored, n) in sorted(worst.items()):
        terminalreporter.write_line("  %.3e  %d / %d  %d  %s" % (rel, judged, floored, n, test))
