import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP path)")
    config.addinivalue_line("markers", "slow: full-size workload, minutes of host work")


@pytest.fixture(scope="session")
def orc():
    import oracle
    return oracle


@pytest.fixture(scope="session")
def wl():
    import workloads
    return workloads


@pytest.fixture(scope="session", autouse=True)
def _progress_lines(request):
    """Progress lines of long GPU tests bypass output capture."""
    import _gpu_common
    _gpu_common.CAPTURE = request.config.pluginmanager.get_plugin("capturemanager")
    yield
    _gpu_common.CAPTURE = None
