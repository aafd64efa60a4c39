import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    # Tests load the in-tree library; build it only when nothing is built yet.
    from paper_2108_03917_amd.lattice import LIB_PATH

    if not os.path.exists(LIB_PATH):
        from paper_2108_03917_amd import _build

        _build.build()
