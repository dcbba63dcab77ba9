import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU oracle runs")


def pytest_collection_modifyitems(config, items):
    # A RuntimeWarning in a GPU test (an invalid cast, an overflow) means the
    # test read memory the library never wrote or computed outside the range
    # it meant to: fail instead of printing it.
    for it in items:
        if "gpu" in it.keywords:
            it.add_marker(pytest.mark.filterwarnings("error::RuntimeWarning"))
    # GPU tests need a device; skip them (with a reason) where none is visible.
    try:
        import torch
        have_gpu = torch.cuda.is_available()
    except Exception:
        have_gpu = False
    if have_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for it in items:
        if "gpu" in it.keywords:
            it.add_marker(skip)
