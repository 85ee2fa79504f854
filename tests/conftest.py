import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built libfastbfp.so")


def pytest_collection_modifyitems(config, items):
    # GPU tests print the case they run before touching the GPU.
    for item in items:
        if item.get_closest_marker("gpu") is not None:
            item.add_marker(pytest.mark.timeout(300))


@pytest.fixture(scope="session")
def host_threads():
    return max(1, min(16, os.cpu_count() or 1))
