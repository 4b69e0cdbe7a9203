import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running statistical test")


@pytest.fixture(scope="session")
def orc():
    from oracle import oracle as o
    o.lib()
    return o


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Reports the near-tie decisions of every GPU-vs-oracle verify comparison
    (the parity bar excludes decisions within 1e-6 of a tie; they are
    counted and printed here)."""
    try:
        from oracle import parity
    except ImportError:
        return
    lines = parity.summary()
    if lines:
        terminalreporter.section("verify parity: near-tie report")
        for l in lines:
            terminalreporter.write_line(l)
