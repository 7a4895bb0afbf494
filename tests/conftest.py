import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (HIP device); parity and GPU property tests")
    config.addinivalue_line("markers", "slow: long CPU-side work")


def pytest_runtest_setup(item):
    # GPU tests read the forward status word after every forward call (a wait
    # that gave up or stale counters fail the test)
    if item.get_closest_marker("gpu") is not None:
        from paper_2607_05583_amd import ops
        ops.CHECK_FWD_STATUS = True
