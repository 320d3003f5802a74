import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size oracle work (minutes of CPU)")


def pytest_collection_modifyitems(config, items):
    # GPU tests run in one process on a machine with the GPU; on one without a
    # GPU they are skipped rather than failing on device allocation.
    try:
        import torch
        have_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        have_gpu = False
    if have_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)


@pytest.fixture(scope="session")
def c1_art():
    """The 9728 -> 2560 down_proj workload (64 decode rows) and its oracle export
    (about 20 s of CPU, computed once per session)."""
    from oracle import prquant as pq
    from paper_2609_22106_amd import inputs
    c = inputs.down_proj_decode()
    return c, pq.prepare(c.W, c.Xcal, 0.5, 256)
