import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


import pytest  # noqa: E402


@pytest.fixture(autouse=True)
def _default_call_opts():
    """Every test starts and ends with the library's default call options (the
    kernel family and wait bound a test may select apply to its thread only)."""
    yield
    mod = sys.modules.get("paper_2605_11111_amd.shardconv")
    if mod is not None:
        mod.shard_set_call_opts()
