import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    # The oracle's library is (re)built here if it is missing or stale: this hook runs
    # before anything initialises the GPU, and no process that has touched the GPU may
    # start the compiler.
    from oracle import build as obuild
    obuild.ensure_built()


def pytest_collection_modifyitems(config, items):
    # A GPU test on a machine without a GPU is skipped (never silently run elsewhere).
    try:
        import torch
        # counting devices does not initialise the GPU runtime in this process
        has_gpu = torch.cuda.device_count() > 0
    except Exception:  # pragma: no cover
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)
