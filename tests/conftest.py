import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the HIP C-ABI library)")


import pytest  # noqa: E402


@pytest.fixture(autouse=True)
def _planner_defaults():
    """Every test starts and ends with the planner's own choices (tests that force a split
    or a work order set them through csr_set_plan_overrides) and with the profiling hooks off."""
    yield
    from paper_2605_07325_amd import csr

    if csr._lib is not None:
        csr.set_plan_overrides()
        csr.set_workgroup_clock(None)
        csr.set_attention_events(None, None)
