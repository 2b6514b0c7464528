import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: runs the HIP path on an MI355X through the C ABI")
    config.addinivalue_line("markers", "slow: long CPU test")


@pytest.fixture(autouse=True)
def _gpu_test_bookkeeping(request):
    """GPU tests: name the test for the parity tallies it creates and, after
    it, require every live model's enqueued work to have finished without an
    asynchronous error or a sticky device error bit (m2r2_sync_check)."""
    if request.node.get_closest_marker("gpu") is None:
        yield
        return
    from tests import gpu_harness as gh
    gh.CURRENT_TEST[0] = request.node.nodeid
    print(f"[gpu test] {request.node.nodeid}", file=sys.stderr, flush=True)
    yield
    for m in gh.live_models():
        m.sync_check()   # raises on an asynchronous HIP error or a sticky device error bit


def pytest_terminal_summary(terminalreporter):
    gh = sys.modules.get("tests.gpu_harness")
    if gh is None or not gh.TALLIES:
        return
    tr = terminalreporter
    tr.write_sep("-", "parity tallies (decisions compared / skipped, arrays, full steps, worst errors)")
    for nodeid, t in gh.TALLIES:
        name = (nodeid or "?").split("::", 1)[-1]
        tr.write_line(f"{name:70s} dec {t.compared:5d} skip {t.skipped:3d} arr {t.arrays:5d} steps {t.steps:3d} "
                      f"worst {t.worst:.2e} elem {t.worst_elem:.2e}")
