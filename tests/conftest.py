import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(autouse=True)
def guard_bands(request):
    """For every GPU test, every output and workspace the binding allocates
    sits between guard bands, checked after the test's calls."""
    if request.node.get_closest_marker("gpu") is None:
        yield None
        return
    from guard import GuardedAllocator
    from paper_2609_37581_amd import trevs
    alloc = GuardedAllocator()
    prev = trevs.set_allocator(alloc)
    try:
        yield alloc
    finally:
        trevs.set_allocator(prev)
    alloc.check()
