import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

_PARITY_KEY = pytest.StashKey[dict]()


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU; calls the HIP library")
    config.stash[_PARITY_KEY] = {}


@pytest.fixture
def record_parity(request):
    """Record the achieved error of a parity case; printed in the terminal summary."""
    def rec(name, **values):
        request.config.stash[_PARITY_KEY][name] = values
    return rec


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    log = config.stash.get(_PARITY_KEY, {})
    if not log:
        return
    terminalreporter.write_sep("-", "achieved parity against the fp64 oracle")
    for name in sorted(log):
        vals = ", ".join(f"{k} {v:.3e}" if isinstance(v, float) else f"{k} {v}" for k, v in log[name].items())
        terminalreporter.write_line(f"{name}: {vals}")
