"""Shared test set-up: the ``gpu`` marker and the CPU-side libraries."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the HIP library")


@pytest.fixture(scope="session", autouse=True)
def _cpu_libs():
    """Compile the oracle and the input generator once if they are not built yet."""
    import lsgen
    import oracle
    lsgen.build(force=False)
    oracle.build(force=False)
