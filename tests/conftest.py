"""Shared pytest configuration.

Markers: ``gpu`` tests need an MI355X (gfx950) and the built HIP library; every
other test runs on the CPU.  The CPU oracle (``oracle/``) is test
infrastructure and is rebuilt here once per session when its source is newer
than its shared object.
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session", autouse=True)
def _oracle_built():
    import oracle
    oracle.build(force=False)
    yield
