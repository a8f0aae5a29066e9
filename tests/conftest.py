import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library on cuda:0)")
    config.addinivalue_line("markers", "big: full-size model shapes (minutes on an MI355X)")


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


_MODEL_ORDER = {"7b": 0, "13b": 1, "70b": 2}


def pytest_collection_modifyitems(config, items):
    """Full-shape tests run grouped by model, so each model is built once."""
    big = [i for i, it in enumerate(items) if it.get_closest_marker("big")]
    if not big:
        return
    group = [items[i] for i in big]
    group.sort(key=lambda it: _MODEL_ORDER.get(getattr(getattr(it, "callspec", None), "params", {}).get("name"), 9))
    for i, it in zip(big, group):
        items[i] = it
