import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture
def tune():
    """Planner overrides for one test: ``tune(GEMV_KIND=2)``; every value set is restored
    when the test ends (through lutgemm_set_tuning, not the environment)."""
    import paper_2408_06003_amd as L
    saved = {}

    def set_(**kw):
        for k, v in kw.items():
            if k not in saved:
                saved[k] = L.get_tuning(k)
            L.set_tuning(k, int(v))

    yield set_
    for k, v in saved.items():
        L.set_tuning(k, v)
