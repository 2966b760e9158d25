import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """One line per GPU parity comparison (rule, errors, excused ties,
    samples compared end to end), so that the figures appear in the session
    output even under -q."""
    mod = sys.modules.get("tests.gpu_util")
    lines = getattr(mod, "PARITY_LOG", None) if mod else None
    if lines:
        terminalreporter.section("parity summary")
        for line in lines:
            terminalreporter.write_line(line)
