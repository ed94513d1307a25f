import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: large workload, minutes of CPU time")


def pytest_terminal_summary(terminalreporter):
    helpers = sys.modules.get("parity_helpers")
    if helpers is not None and getattr(helpers, "MAX_ERR", None):
        items = ", ".join(f"{k} {v:.2e}" for k, v in sorted(helpers.MAX_ERR.items()))
        terminalreporter.write_line(f"max |gpu - oracle| per check: {items}")
