import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
# Host-only tests pass made-up device addresses to entry points whose checks
# they expect to pass; without a GPU the launch then fails with a status, with
# one it would read those addresses. Such calls run only where no GPU exists.
GPU_PRESENT = os.path.exists("/dev/kfd")
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test")


def _gpu_tests_selected(config) -> bool:
    expr = (config.getoption("markexpr", "") or "").replace(" ", "")
    return expr != "notgpu"


def pytest_sessionstart(session):
    # The full-size parity tests run the oracle on worker processes. Their fork
    # server starts here, before any test touches the GPU, so no worker is ever
    # forked from a process that has initialised the GPU.
    if _gpu_tests_selected(session.config):
        from oracle import ranges
        ranges.start_forkserver()
