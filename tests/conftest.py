import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size parity cases (tens of seconds)")


def _ensure_host_libs():
    """Build the CPU-side libraries if nothing is built yet (never rebuilds)."""
    import oracle
    from paper_2510_13161_amd import synth
    from paper_2510_13161_amd import build as pkg_build
    if not os.path.exists(oracle.LIB_PATH):
        oracle.build()
    if not os.path.exists(synth.HOST_LIB):
        pkg_build.build_synth_host()


@pytest.fixture(scope="session", autouse=True)
def host_libs():
    _ensure_host_libs()
