import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    # Build the library only when nothing is built yet (after a source
    # change, build again explicitly: __graft_entry__.build()).
    if not os.path.exists(os.path.join(ROOT, "paper_2609_34334_amd", "libhoccl.so")):
        import __graft_entry__
        __graft_entry__.build()


import pytest  # noqa: E402


@pytest.fixture(autouse=True)
def _ring_unless_asked():
    """The library's default reduction is AUTO, which folds directly on one
    GPU.  The tests are written for the ring schedule and ask for the fold
    or AUTO explicitly, so every test starts from reduce_algo = ring."""
    import paper_2609_34334_amd as hc
    saved = hc.get_config()
    hc.set_config(reduce_algo="ring")
    yield
    hc.set_config(**saved)
