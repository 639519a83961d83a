import os
import sys

import pytest
import torch  # noqa: F401  (imported at collection: a cold first import is slow)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU-only check")


@pytest.fixture(scope="session")
def gpu_lib():
    """The built HIP library through its Python binding, on a GPU device.
    Fails loudly (no CPU fallback) if the library or the GPU is missing."""
    import torch
    import paper_2507_08784_amd as glr
    if not torch.cuda.is_available():
        pytest.fail("GPU test collected on a machine without a GPU")
    glr.load()  # raises if the shared library was not built
    return glr
