import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")
    config.addinivalue_line("markers", "spawns: starts child processes (CPU only; skipped once this process "
                                       "has initialised the GPU)")


@pytest.hookimpl(tryfirst=True)
def pytest_runtest_setup(item):
    # a process that has initialised the GPU starts no other programs: a run
    # that mixes GPU tests with these leaves them out once the GPU is in use
    if item.get_closest_marker("spawns") is None:
        return
    torch = sys.modules.get("torch")
    if torch is not None and torch.cuda.is_initialized():
        pytest.skip("starts child processes; this process has initialised the GPU")


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    oracle.lib()
    return oracle
