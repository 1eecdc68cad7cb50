import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running case")
    # The float64 oracle's worker pool for the whole-workload comparisons is
    # forked here, before anything in this process touches the GPU.
    if "not gpu" not in (config.getoption("-m") or ""):
        from tests import oracle_pool
        oracle_pool.start()


def pytest_unconfigure(config):
    from tests import oracle_pool
    oracle_pool.close()


def _gpu_available():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def pytest_collection_modifyitems(config, items):
    if _gpu_available():
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)
