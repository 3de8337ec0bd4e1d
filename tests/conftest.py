import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size parity cases (seconds to minutes)")


def gpu_available() -> bool:
    try:
        import torch

        return torch.cuda.is_available()
    except Exception:  # pragma: no cover
        return False


@pytest.fixture(scope="session")
def lib():
    """The loaded C-ABI library (skips when no GPU is present; raises when the build is missing)."""
    if not gpu_available():
        pytest.skip("no GPU")
    from paper_2607_07862_amd import binding

    lib = binding.load()
    # the GPU suite checks the product library, never the timing-trace build
    assert os.path.abspath(binding.loaded_path()) == os.path.abspath(binding.LIB_PATH), binding.loaded_path()
    return lib
