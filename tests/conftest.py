import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU-side oracle run")


@pytest.fixture(scope="session")
def orc():
    from oracle import oracle
    oracle.lib()
    return oracle


def pytest_terminal_summary(terminalreporter):
    """Max-abs error of every parity check of the session (tests/gpu_util.py)."""
    mod = sys.modules.get("gpu_util")
    if mod is None or not getattr(mod, "RESULTS", None):
        return
    terminalreporter.section("parity: max-abs error per tensor (bound: tol + half an ulp of the output type)")
    for label, md, tol, margin in mod.RESULTS:
        terminalreporter.write_line(f"{label:78s} max-abs {md:.3e}  tol {tol:g}  margin {margin:.3e}")
