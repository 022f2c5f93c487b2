import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


import pytest  # noqa: E402


@pytest.fixture(scope="session", autouse=True)
def _oracle_pool_shutdown():
    """Stop the oracle's CPU worker processes (started on first use) at the end of the session."""
    yield
    from tests import oracle_pool
    oracle_pool.close()
