import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def gpu_available():
    import torch
    return torch.cuda.is_available()


def pytest_terminal_summary(terminalreporter):
    """The largest GPU-vs-oracle errors seen by check_step in this run."""
    import sys
    mod = sys.modules.get("tests.parity")
    if mod is not None and any(mod.SEEN.values()):
        terminalreporter.write_line(
            "parity: largest errors seen: " + ", ".join(f"{k} {v:.3g}" for k, v in mod.SEEN.items()))
