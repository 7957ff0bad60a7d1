import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test")


@pytest.fixture(scope="session")
def oracle():
    """The CPU test oracle, rebuilt once per session from its C source."""
    import oracle as _o
    from oracle import build as _b
    src = os.path.join(ROOT, "oracle", "sv_oracle.c")
    if (not os.path.exists(_b.LIB) or os.path.getmtime(_b.LIB) < os.path.getmtime(src)):
        _b.build()
    _o.lib()
    return _o
