import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session", autouse=True)
def _host_libs():
    """The oracle and the input generator are plain C; build them if they are not built yet."""
    import oracle
    import synth

    if not os.path.exists(oracle._LIB_PATH):
        oracle.build()
    if not os.path.exists(synth._LIB_PATH):
        synth.build()
