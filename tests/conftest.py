import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library on cuda:0)")
    config.addinivalue_line("markers", "big: full-size model shapes (minutes; GPU box only)")


@pytest.fixture(scope="session", autouse=True)
def _built_helpers():
    """The C helpers (oracle, input filler) are built once if missing."""
    import oracle
    import sd_synth

    if not os.path.exists(oracle.LIB_PATH):
        oracle.build()
    if not os.path.exists(sd_synth._LIB_PATH):
        sd_synth.build()
    yield
