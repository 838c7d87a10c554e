import os
import sys

import pytest

# The GPU tests run with eight hardware queues per process, like bench.py, so
# libmori's copy-engine swaps use their own copy streams (double-buffered).  The
# in-order variant used with HIP's default of four queues is covered by
# test_gpu_parity.py::test_default_queue_count_in_order_copies.
os.environ["GPU_MAX_HW_QUEUES"] = "8"

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workloads (tens of GiB)")


@pytest.fixture(scope="session")
def orc():
    from oracle import oracle
    oracle.lib()
    return oracle
