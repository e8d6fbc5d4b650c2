import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_sessionstart(session):
    # the tests load the in-tree libsmat.so; build it once if this checkout has none yet
    from paper_2609_33437_amd import build
    if not os.path.exists(build.LIB) and build.hipcc_available():
        build.build()
