import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size parity cases")


@pytest.fixture(autouse=True)
def _gpu_tests_run_on_the_native_path(request):
    """A test marked gpu fails, rather than skips or passes, when no GPU is
    visible or the HIP library cannot be loaded."""
    if request.node.get_closest_marker("gpu") is not None:
        import torch
        assert torch.cuda.is_available(), "GPU test without a visible GPU"
        from paper_2608_15797_amd import kvr  # noqa: F401  (raises when libkvr.so is missing)
    yield
