import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers",
                            "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_terminal_summary(terminalreporter):
    # the count-parity figures of the GPU tests (tie-band exemptions, differing rows)
    mod = sys.modules.get("parity_util")
    lines = mod.count_summary() if mod is not None else []
    if lines:
        terminalreporter.write_sep("-", "retained-tile count parity")
        for ln in lines:
            terminalreporter.write_line(ln)


@pytest.fixture(scope="session")
def gpu_available():
    import torch
    return torch.cuda.is_available()
