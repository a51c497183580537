import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    # the CPU libraries are cheap to build; build them when absent so the CPU suite is self-contained
    import __graft_entry__ as ge
    ge.build_cpu_libs(only_missing=True)


@pytest.fixture(scope="session")
def gpu_lib():
    """The HIP library, loaded through its binding; fails loudly when unusable."""
    import torch

    if not torch.cuda.is_available():
        pytest.fail("GPU test selected but no GPU is visible")
    from paper_2608_15437_amd import mmbev

    mmbev.load()
    return mmbev
