import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")


@pytest.fixture(scope="session")
def gpu_ctx():
    """One library context on cuda:0 for the whole GPU session."""
    import torch
    from paper_2407_00051_amd import Context
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ctx = Context(0)
    yield ctx
    ctx.close()
