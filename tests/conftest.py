import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an AMD MI355X (gfx950) GPU and the built HIP library")


def pytest_runtest_setup(item):
    if "parity" in sys.modules:
        sys.modules["parity"].CURRENT["test"] = item.nodeid


def pytest_terminal_summary(terminalreporter):
    """Raw max-abs error of every compared tensor, with its bf16 floor where one applies."""
    par = sys.modules.get("parity")
    if par is None or not par.RECORDS:
        return
    terminalreporter.section("parity: raw max-abs errors against the oracle")
    for line in par.summary_lines():
        terminalreporter.write_line(line)
    path = os.environ.get("LH_PARITY_JSON")
    if path:
        os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
        with open(path, "w") as fh:
            json.dump(par.RECORDS, fh)


@pytest.fixture(scope="session")
def rng():
    import numpy as np
    return np.random.default_rng(12345)
