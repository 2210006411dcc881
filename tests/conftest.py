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
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(autouse=True)
def _unchecked_library(monkeypatch):
    """Every test starts with the library's checked mode off, whatever the
    environment says: several tests feed the fast path hostile tables on
    purpose to see its silent skips, which checked mode would refuse.  Tests
    of checked mode switch it on themselves."""
    monkeypatch.delenv("TOPKV_CHECKED", raising=False)
