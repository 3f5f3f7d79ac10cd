import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: longer CPU test")
    # The oracle's process pool forks from a server started now, before any
    # test initialises the GPU (GPU runs only).
    if "not gpu" not in (config.getoption("markexpr") or "").replace("  ", " "):
        from tests import oracle_pool
        oracle_pool.start()


@pytest.fixture(autouse=True)
def _announce_gpu_case(request):
    """Name every GPU case on stdout before it runs (attributes a fault to its case)."""
    if request.node.get_closest_marker("gpu") is not None:
        print(f"\n[gpu-case] {request.node.nodeid}", flush=True)
    yield
