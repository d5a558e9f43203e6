import os
import sys

import time

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


@pytest.fixture(scope="session")
def gpu():
    """Skip unless a ROCm GPU is present; returns the torch device."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.fixture
def progress(capsys):
    """Report a long test's steps as they finish, past pytest's output capture
    (a run that prints nothing for minutes is taken to be hung), with the
    seconds since the test started."""
    t0 = time.monotonic()

    def say(msg):
        with capsys.disabled():
            print(f"[{time.monotonic() - t0:6.1f}s] {msg}", flush=True)
    return say
