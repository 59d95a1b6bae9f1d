import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


@pytest.fixture(params=[1, 2], ids=["scattered", "streaming"])
def apply_form(request):
    """Runs a server-apply test under each form of the apply (1: scattered, 2: streaming wherever the
    parameters are 16-byte aligned), then restores the per-call choice."""
    from paper_1704_05021_amd import gd
    gd.debug_apply_form(request.param)
    yield request.param
    gd.debug_apply_form(0)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workloads (seconds of CPU work each)")
