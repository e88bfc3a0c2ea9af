import os
import subprocess
import sys

import pytest

TESTS = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(TESTS)
for _p in (ROOT, TESTS):
    if _p not in sys.path:
        sys.path.insert(0, _p)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) HIP device")


def _ensure_oracle_built():
    lib = os.path.join(ROOT, "oracle", "libws_oracle.so")
    if not os.path.exists(lib):
        subprocess.run([sys.executable, os.path.join(ROOT, "oracle", "build.py")], check=True)


_ensure_oracle_built()


def gpu_available():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def ws():
    """The HIP library binding (built on demand when nothing is built)."""
    if not gpu_available():
        pytest.skip("no HIP device")
    from paper_2607_04443_amd import _build
    if not os.path.exists(_build.LIB_PATH):
        _build.build()
    from paper_2607_04443_amd import ws as wsmod
    return wsmod
