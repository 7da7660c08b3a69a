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
