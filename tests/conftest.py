import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter):
    """Worst error of every GPU parity check of the session, per test: output
    max-abs (gate 2e-2) and the worst (sequence, head) state relative
    Frobenius error (gate 1e-3)."""
    mod = sys.modules.get("gpu_helpers")
    rows = getattr(mod, "RESULTS", None) if mod is not None else None
    if not rows:
        return
    worst = {}
    for test, check, what, err in rows:
        key = (test, check)
        worst[key] = max(worst.get(key, 0.0), err)
    terminalreporter.write_sep("-", "GPU parity: worst error per test")
    for (test, check), err in sorted(worst.items()):
        terminalreporter.write_line(f"{test}  {check} {err:.3e}")
