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
def _host_libs():
    """The oracle and the workload generators are plain C; build them if absent or stale."""
    from oracle import oracle
    from paper_2407_15264_amd import workload
    if oracle.stale():
        oracle.build()
    if not os.path.exists(workload.LIB_PATH):
        workload.build()
