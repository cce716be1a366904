import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def gpu_lib():
    """The loaded HIP library, on a machine with a GPU.  Fails loudly if the
    library is missing: GPU tests never fall back to another implementation."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test collected on a machine without a GPU")
    from paper_2609_33503_amd import relaxkv
    return relaxkv.load()


@pytest.fixture(scope="session")
def rk():
    """The binding with the in-tree library loaded for host-only calls (built
    first when it is missing or stale; CPU tests never launch kernels)."""
    from paper_2609_33503_amd import build, relaxkv
    try:
        build.verify()
    except RuntimeError:                             # missing or stale: build it (CPU only)
        build.build()
    relaxkv.load()
    return relaxkv
