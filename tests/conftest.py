import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def _ensure_built():
    # Load what is built; build only when a library is missing.
    import oracle.build
    import tracegen.build
    if not os.path.exists(oracle.build.LIB):
        oracle.build.build()
    if not os.path.exists(tracegen.build.LIB):
        tracegen.build.build()


_ensure_built()


@pytest.fixture(scope="session")
def tiny_trace():
    import tracegen
    return tracegen.make("tiny")
