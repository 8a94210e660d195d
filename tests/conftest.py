import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


import pytest  # noqa: E402


@pytest.fixture
def knob():
    """Sets tuning overrides of the library (ds_set_tuning) for one test and
    restores their previous values afterwards: knob("DS_FORCE_VARIANT", 0)."""
    from paper_1905_13298_amd import ops
    saved = {}

    def set_(name, value):
        if name not in saved:
            saved[name] = ops.get_tuning(name)
        ops.set_tuning(name, value)

    yield set_
    for name, value in saved.items():
        ops.set_tuning(name, value)
