import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built libpkv")
    config.addinivalue_line("markers", "slow: large CPU work")


@pytest.fixture(scope="session")
def repo_root():
    return ROOT


def pytest_collection_finish(session):
    """GPU runs: fork the suffix-row draw workers before any test touches the GPU."""
    if any(item.get_closest_marker("gpu") for item in session.items):
        from paper_2609_26219_amd import device
        device.start_workers()
