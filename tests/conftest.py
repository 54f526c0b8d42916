import os
import sys

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if REPO not in sys.path:
    sys.path.insert(0, REPO)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library"
    )


@pytest.fixture(scope="session")
def gpu_lib():
    """The HIP library loaded through the binding, on a visible GPU.

    A GPU test fails (it does not skip) when no GPU is visible or the built
    library is missing: a silent fallback would hide a broken build.
    """
    import torch

    if not torch.cuda.is_available():
        pytest.fail("GPU test selected but torch sees no GPU")
    import paper_1412_7091_amd as lst

    lst.load_library()
    return lst
