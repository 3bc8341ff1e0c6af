import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU-only check")


def pytest_collection_modifyitems(config, items):
    # keep the full-size GPU cases after the small ones so a failure in a small
    # case stops ``-x`` before the expensive ones start; the allocation-free
    # entry point's test runs last of all
    def order(it):
        if "test_zz_" in it.nodeid:
            return 2
        return 1 if "fullsize" in it.nodeid else 0

    items.sort(key=order)
