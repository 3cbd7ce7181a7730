import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


import pytest


@pytest.fixture(autouse=True)
def _clear_plan_overrides():
    """Planner overrides are process-wide: every test starts and ends without."""
    yield
    try:
        from paper_2608_28003_amd import w8a8
    except Exception:
        return
    if w8a8._lib is not None:
        w8a8.clear_plan_overrides()
