import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: large host-memory or long-running case")


@pytest.fixture(scope="session")
def orc():
    import oracle
    return oracle.default()


@pytest.fixture(autouse=True)
def _release_device_memory(request):
    """After each GPU test, hand the device memory PyTorch's caching allocator
    kept back to the driver. Freeing very large allocations (the 70B and
    many-tile tests hold up to 282 GB) starts work in the driver that slows
    pageable host-to-device loads for some seconds; doing it as each test
    ends, rather than all at once when the process exits, keeps that away
    from whatever runs next."""
    yield
    if request.node.get_closest_marker("gpu") is None:
        return
    import gc
    gc.collect()
    torch = sys.modules.get("torch")
    if torch is not None and torch.cuda.is_available():
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
