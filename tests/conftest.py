import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library)")
    config.addinivalue_line("markers", "forces_give_up: a GPU test that makes exchange waits "
                                       "give up on purpose (host-set wait limit)")


@pytest.fixture(autouse=True)
def _no_exchange_give_ups(request):
    """Every GPU test that does not force them checks that no exchange wait
    of the split forms gave up while it ran (rowsm_split_wait_failures()
    synchronises the device and reads the device's cumulative count)."""
    if (request.node.get_closest_marker("gpu") is None
            or request.node.get_closest_marker("forces_give_up") is not None
            or not _gpu_available()):
        yield
        return
    import paper_2607_23089_amd as R
    before = R.rowsm_split_wait_failures()
    yield
    after = R.rowsm_split_wait_failures()
    assert before >= 0 and after == before, \
        f"exchange waits gave up during the test ({before} -> {after})"


def _gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def pytest_collection_modifyitems(config, items):
    if _gpu_available():
        return
    skip = pytest.mark.skip(reason="no GPU in this environment")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)
