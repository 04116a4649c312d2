import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def _ensure_built():
    """Builds the CPU-side libraries if they are missing (GPU code is built by
    __graft_entry__.build() beforehand and only loaded here)."""
    from oracle import build as ob
    from synth import build as sb
    if not os.path.exists(os.path.join(ROOT, "oracle", "liboracle.so")):
        ob.build()
    if not os.path.exists(os.path.join(ROOT, "synth", "libsynth_cpu.so")):
        sb.build_cpu()


_ensure_built()


@pytest.fixture(scope="session")
def root():
    return ROOT
