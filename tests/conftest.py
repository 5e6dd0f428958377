import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_sessionstart(session):
    """Build libtim.so once if it is not there (hipcc cross-compiles without a GPU)."""
    lib = os.path.join(ROOT, "paper_2605_14220_amd", "libtim.so")
    if not os.path.exists(lib):
        from paper_2605_14220_amd.build import build
        build()
