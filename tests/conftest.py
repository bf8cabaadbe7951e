import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session", autouse=True)
def _oracle_built():
    """The oracle library is test infrastructure; build it if missing."""
    lib = os.path.join(ROOT, "oracle", "liboracle.so")
    if not os.path.exists(lib):
        from oracle import build
        build.build()
    yield


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Print what the full-size parity tests compared (also under -q)."""
    from tests import parity
    if parity.COVERAGE:
        terminalreporter.section("parity coverage")
        for line in parity.COVERAGE:
            terminalreporter.write_line(line)
