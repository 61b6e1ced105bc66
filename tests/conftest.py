"""Shared test configuration.

``-m gpu`` tests need an MI355X (gfx950) and the built HIP library; every
other test runs on the CPU.
"""
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
for p in (ROOT, ROOT / "tests"):
    if str(p) not in sys.path:
        sys.path.insert(0, str(p))


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def orc():
    import oracle
    o = oracle.load()
    # a library loaded into this process may have switched on flush-to-zero
    assert o.selfcheck() == 0, "floating-point environment changed (FTZ/DAZ?)"
    return o
