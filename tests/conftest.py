import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def _ensure_built():
    """Load what is built; build only what is missing (hipcc cross-compiles on CPU)."""
    from oracle import build as ob
    if not os.path.exists(ob.LIB):
        ob.build()
    from synth import build as sb
    if not os.path.exists(sb.LIB):
        sb.build()
    if os.path.exists(os.path.join(ROOT, "paper_2607_05804_amd", "_build.py")):
        from paper_2607_05804_amd import _build as pb
        if not os.path.exists(pb.LIB):
            pb.build()


_ensure_built()


@pytest.fixture(scope="session")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test collected on a machine without a GPU")
    return torch.device("cuda:0")
