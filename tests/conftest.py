import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def root():
    return ROOT


def pytest_sessionfinish(session, exitstatus):
    # the parity measurements of this session (tests/parity.py), when asked for
    path = os.environ.get("TABPACK_PARITY_REPORT")
    if path:
        import parity
        parity.dump_records(path)
