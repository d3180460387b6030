import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# HIP multiplexes a process's streams onto GPU_MAX_HW_QUEUES hardware queues
# (4 by default); streams that share a queue run its packets in order, so a
# stream waiting for an event, or a long kernel, also holds back the other
# streams on that queue.  The readiness tests run about ten streams at once
# (the library's, the dispatch streams, a delayed stream): one queue each.
# Read when HIP initialises, i.e. before any test touches the GPU.
os.environ["GPU_MAX_HW_QUEUES"] = "16"


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workload; minutes on the CPU")
