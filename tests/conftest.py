import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs a gfx950 GPU (runs through the C-ABI)")
    config.addinivalue_line("markers", "slow: full-size parity cases")


@pytest.fixture
def tune():
    """Force the walks' launch plan (tune(split=..., group=..., waves=...,
    nbuf=..., chunk=...)) or the layout of later loads (tune(layout=...))
    through the library's tuning entry points; restores the planner's and
    loader's choices afterwards."""
    from paper_2411_10764_amd import ml2
    plan = {}

    def force(layout=None, **kw):
        if layout is not None:
            ml2.ml2_tune_layout(layout)
        if kw:
            plan.update({k: int(v) for k, v in kw.items()})
            ml2.ml2_tune_walk_plan(**plan)

    yield force
    ml2.ml2_tune_walk_plan()
    ml2.ml2_tune_layout(0)
