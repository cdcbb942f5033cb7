import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: longer CPU test")


import pytest


@pytest.fixture(autouse=True)
def _reset_schedule_overrides():
    """Every test starts and ends with the library's own schedule choices
    (lce_set_tuning overrides are process-wide)."""
    yield
    mod = sys.modules.get("paper_2011_09398_amd")
    if mod is not None and getattr(mod, "_lib", None) is not None:
        mod.set_tuning(**{k: 0 for k in mod.TUNING_KEYS})
