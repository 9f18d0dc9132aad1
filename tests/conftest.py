import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def golden_dir():
    return os.path.join(ROOT, "tests", "golden")


@pytest.fixture
def overrides(monkeypatch):
    """monkeypatch with the library's tuning overrides switched on
    (CAFFE_PROFILE_OVERRIDES=1): tests that force a kernel variant, tile or
    split count set the CAFFE_* variables through it."""
    monkeypatch.setenv("CAFFE_PROFILE_OVERRIDES", "1")
    return monkeypatch
