import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def gpu_available():
    import torch
    return torch.cuda.is_available()


def pytest_sessionfinish(session, exitstatus):
    # per-call parity statistics (max |g - r|, elements above the flat bound),
    # written only when SDATTN_PARITY_REPORT names a file
    try:
        import parity_util
    except ImportError:
        return
    parity_util.write_report()
