import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running case")


# The 256K stack layers are drawn and run through the oracle's estimation
# stages in spawned processes that start at the end of collection, before any
# test touches the GPU (tests/pregen.py).
STACK_TEST = "test_256k_layer_sampled_rows"
STACK_ROWS_PER_HEAD = 512


def pytest_collection_finish(session):
    seeds = sorted({item.callspec.params["layer"] for item in session.items
                    if getattr(item, "originalname", "") == STACK_TEST})
    if not seeds:
        return
    try:
        import torch
        if torch.cuda.device_count() == 0:     # counts devices without initialising them
            return
    except ImportError:
        return
    from tests import pregen
    pregen.start(seeds, STACK_ROWS_PER_HEAD)


def pytest_unconfigure(config):
    try:
        from tests import pregen
    except ImportError:
        return
    pregen.stop()
