import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def golden():
    import json
    with open(os.path.join(ROOT, "tests", "golden", "worked_examples.json")) as f:
        return json.load(f)


def pytest_terminal_summary(terminalreporter):
    """Every parity figure of the session (per-head Frobenius ratio and the
    element-wise |gpu - ref| / (|ref| + rms(ref row))), passing or not."""
    parity = sys.modules.get("parity")
    if parity is None or not parity.RECORD:
        return
    terminalreporter.section("parity figures (frob / elem vs tolerance)")
    for tag, name, frob, elem, tol in parity.RECORD:
        terminalreporter.write_line(f"{tag:48.48s} {name:3s} frob {frob:.2e} elem {elem:.2e} tol {tol:.0e}")
