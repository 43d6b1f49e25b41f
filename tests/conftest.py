import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long CPU test")


import pytest  # noqa: E402


@pytest.fixture(scope="session")
def lib():
    """The built C library; built once here only if no build exists yet."""
    from paper_2010_14109_amd import ooc
    if not os.path.exists(ooc.LIB_PATH):
        from paper_2010_14109_amd import build
        build.build()
    return ooc.load()
