import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session", autouse=True)
def _synth_built():
    """The generator library is plain C; build it once if it is missing."""
    from synth import build as sb
    if not os.path.exists(os.path.join(ROOT, "synth", "libsynth.so")):
        sb.build()
    yield


def golden_path(name):
    return os.path.join(ROOT, "tests", "golden", name)
