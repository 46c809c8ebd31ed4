import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_sessionfinish(session, exitstatus):
    # per-tensor parity margins (max abs, relative L2, worst error over its
    # bound) of every comparison the session made
    import _util
    path = os.environ.get("DM_PARITY_MARGINS", os.path.join(ROOT, "gpurun_out", "parity_margins.json"))
    _util.write_margins(path)
