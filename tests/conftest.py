import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# The library is built in-tree; build it only when nothing is there yet.
_LIB = os.path.join(ROOT, "paper_2410_12982_amd", "liblcsm.so")
if not os.path.exists(_LIB):
    from paper_2410_12982_amd.build import build as _build
    _build()


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
