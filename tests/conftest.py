import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(autouse=True, scope="module")
def _release_gpu_memory():
    """Return each module's cached device memory to the driver when the module ends. torch's caching
    allocator otherwise keeps every block (about 110 GB after the index-limit test) until the process
    exits, and the driver's handling of that much freed memory slows the GPU for a second or two."""
    yield
    torch = sys.modules.get("torch")
    if torch is not None and torch.cuda.is_initialized():
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
