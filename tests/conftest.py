import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running test")


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle
    oracle.build(force=False)
    return oracle


@pytest.fixture(params=[8, 16], ids=["sw8", "sw16"])
def slice_width(request):
    """Runs a GPU test with each scan slice width forced, then restores the automatic choice."""
    from paper_2607_07386_amd import sdm
    sdm.set_scan_slice_width(request.param)
    yield request.param
    sdm.set_scan_slice_width(0)
