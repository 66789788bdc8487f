import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workload (seconds of CPU for inputs/oracle)")


def pytest_collection_modifyitems(config, items):
    # Run GPU tests only when a GPU is actually present; the CPU suite deselects them with -m.
    pass
