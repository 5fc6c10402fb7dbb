import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def _gpu_present():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def pytest_collection_modifyitems(config, items):
    # gpu tests are skipped (never passed) on hosts without a GPU; on a GPU
    # host they call the HIP library and fail loudly if it is missing.
    if any(item.get_closest_marker("gpu") for item in items) and not _gpu_present():
        skip = pytest.mark.skip(reason="no GPU on this host")
        for item in items:
            if item.get_closest_marker("gpu"):
                item.add_marker(skip)
