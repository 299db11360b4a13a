import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session")
def repo_root():
    return ROOT


# Parity checks record one line each (workload, requests, max and mean absolute
# error against the oracle); the lines are printed after the test summary, so
# they appear in quiet runs too.
PARITY_LINES: list = []


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    if PARITY_LINES:
        terminalreporter.section("parity against the fp64 oracle")
        for line in PARITY_LINES:
            terminalreporter.write_line(line)
