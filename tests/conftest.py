import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def _ensure_host_libs():
    # Build the host-side helpers only when nothing is built yet.
    if not os.path.exists(os.path.join(ROOT, "oracle", "liboracle.so")):
        from oracle import build as ob
        ob.build()
    if not os.path.exists(os.path.join(ROOT, "gspn_inputs", "libgspn_inputs.so")):
        from gspn_inputs import build as gb
        gb.build()


_ensure_host_libs()
