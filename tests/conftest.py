import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU-heavy oracle runs (minutes)")


def pytest_collection_modifyitems(config, items):
    # keep GPU tests in the order the files define; nothing to reorder for CPU tests
    pass


@pytest.fixture(scope="session")
def torch_cpu():
    import torch
    torch.set_num_threads(max(1, min(16, len(os.sched_getaffinity(0)))))
    return torch
