import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

LIB = os.path.join(ROOT, "paper_2509_04719_amd", "liborch.so")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU case")


@pytest.fixture(scope="session")
def orch_lib():
    """The ctypes binding of liborch.so; built in-tree only if absent."""
    if not os.path.exists(LIB):
        from paper_2509_04719_amd import build
        build.build()
    from paper_2509_04719_amd import _lib
    return _lib
