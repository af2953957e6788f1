import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workload, minutes of host time")


def pytest_collection_modifyitems(config, items):
    # GPU tests run in file order after the CPU tests so that a GPU failure under
    # `pytest -x` does not hide the host-side results.
    items.sort(key=lambda it: 1 if it.get_closest_marker("gpu") else 0)
