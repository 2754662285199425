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

    # another build of the same library (the AddressSanitizer build of the
    # ABI tests) can be named through DUO_TEST_LIB
    if os.environ.get("DUO_TEST_LIB"):
        duo.LIB_PATH = os.environ["DUO_TEST_LIB"]
        return duo
    if not os.path.exists(duo.LIB_PATH):
        from paper_2506_20194_amd import build

        build.build()
    return duo
