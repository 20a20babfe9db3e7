import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def orc():
    import oracle

    return oracle.load()


@pytest.fixture(autouse=True)
def _no_handover_giveups(request):
    """After every GPU test: no fused hand-over wait gave up (a give-up means a
    launch may have computed with incomplete producer rows)."""
    yield
    if request.node.get_closest_marker("gpu") is None:
        return
    import paper_2606_19528_amd as lm

    n = lm.handover_giveups(reset=True)
    assert n == 0, f"{n} fused hand-over waits gave up during this test"
