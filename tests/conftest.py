import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workload (minutes of oracle time)")


@pytest.fixture(scope="session", autouse=True)
def _oracle_built():
    import oracle
    oracle.build(force=False)
    # a differently built copy of the oracle (the sanitizer run points the pins at one)
    if os.environ.get("HARL_ORACLE_LIBRARY"):
        oracle.use_library(os.environ["HARL_ORACLE_LIBRARY"])
    yield
