import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_sessionstart(session):
    """Build libpvlm.so once if this checkout has none yet (an existing build is
    used as it is; rebuild after changing a source)."""
    lib = os.path.join(ROOT, "paper_2603_19610_amd", "libpvlm.so")
    if not os.path.exists(lib):
        from paper_2603_19610_amd import build as _build
        _build.build(verbose=True)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def gpu_available():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def golden_dir():
    return os.path.join(ROOT, "tests", "golden")
