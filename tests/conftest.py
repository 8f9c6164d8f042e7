"""Shared pytest setup: marker registration, repo root on sys.path, and the
CPU-side builds (generator + oracle) that every test needs."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running (large workloads)")


@pytest.fixture(scope="session", autouse=True)
def _cpu_builds():
    import oracle
    import synth

    synth.build(force=False)
    oracle.build(force=False)
    yield
