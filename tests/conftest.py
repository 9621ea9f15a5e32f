import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def _build_missing():
    """Build the oracle and the HIP library only when nothing is built yet."""
    if not os.path.exists(os.path.join(ROOT, "oracle", "liboracle.so")):
        from oracle import build as ob
        ob.build()
    if not os.path.exists(os.path.join(ROOT, "paper_2512_16473_amd", "libmoe.so")):
        sys.path.insert(0, os.path.join(ROOT, "paper_2512_16473_amd"))
        import build as lb  # paper_2512_16473_amd/build.py
        lb.build()


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")
    _build_missing()


@pytest.fixture(scope="session")
def golden_dir():
    return os.path.join(ROOT, "tests", "golden")
