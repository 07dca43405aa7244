import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TESTS = os.path.dirname(os.path.abspath(__file__))
for p in (ROOT, TESTS):
    if p not in sys.path:
        sys.path.insert(0, p)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_sessionstart(session):
    # The CPU suite checks the library's exports and host-only logic; build it
    # in-tree if it is missing (a GPU run uses the library shipped with the tree).
    lib = os.path.join(ROOT, "paper_2606_15453_amd", "libstmoe.so")
    if not os.path.exists(lib):
        from paper_2606_15453_amd.build import build
        build()
