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


@pytest.fixture(autouse=True)
def _debug_checks_clean(request):
    """With MLSTM_EXPECT_DEBUG_CHECKS=1 (a run on the bounds-checked library, libmlstm_debug.so), every
    GPU test must leave the library's debug flags clear: no computed index left its extent."""
    yield
    if os.environ.get("MLSTM_EXPECT_DEBUG_CHECKS") != "1" or request.node.get_closest_marker("gpu") is None:
        return
    import torch

    from paper_2503_13427_amd import binding

    torch.cuda.synchronize()
    flags = binding.mlstm_debug_flags()
    assert flags == 0, f"device bounds checks failed: flags {flags:#x}"
