import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: large CPU-side oracle work")


@pytest.fixture(scope="session")
def rng_seed():
    return 1234


@pytest.fixture(scope="session")
def duo_lib():
    """The built library; builds it once if it is missing."""
    from paper_2506_20194_amd import duo

    if not os.path.exists(duo.LIB_PATH):
        from paper_2506_20194_amd import build

        build.build()
    return duo
