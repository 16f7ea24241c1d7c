import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: large inputs, minutes of CPU time")
    # Host libraries are built on demand only when nothing is built yet.
    from oracle import build as ob
    from synth import build as sb
    if not os.path.exists(os.path.join(ROOT, "oracle", "libggref.so")):
        ob.build()
    if not os.path.exists(os.path.join(ROOT, "synth", "libsynth.so")):
        sb.build()


@pytest.fixture(scope="session")
def root():
    return ROOT
