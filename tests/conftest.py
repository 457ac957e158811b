import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: larger CPU cases")


def pytest_terminal_summary(terminalreporter):
    """Print the error margins of the whole-output parity checks."""
    mod = sys.modules.get("vda_testutil")
    recs = getattr(mod, "ERROR_RECORDS", None) if mod else None
    if recs:
        terminalreporter.write_line("parity margins against the oracle:")
        for case, rep in recs:
            terminalreporter.write_line(f"  {case}: {rep}")
