import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test")


@pytest.fixture(scope="session", autouse=True)
def _built_cpu_libs():
    """The generator and oracle are plain C; build them if missing."""
    import oracle
    import workload
    if not os.path.exists(workload._SO):
        workload.build()
    if not os.path.exists(oracle._SO):
        oracle.build()
    yield
