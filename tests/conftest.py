import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (runs through the HIP library)")


@pytest.fixture(scope="session")
def gpu_ctx():
    """A library context on cuda:0 (GPU tests only)."""
    import torch
    from paper_2609_13592_amd import binding as bd
    assert torch.cuda.is_available(), "GPU test without a GPU"
    torch.cuda.init()
    ctx = bd.boost_init(0)
    yield ctx
    torch.cuda.synchronize()
    bd.boost_shutdown(ctx)
