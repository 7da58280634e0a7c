import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built libeb.so")


@pytest.fixture(scope="session")
def oracle():
    from oracle import oracle as O

    return O.get()


def pytest_terminal_summary(terminalreporter):
    """Worst normalised error per parity-check label of the GPU tests."""
    mod = sys.modules.get("tests.gpu_helpers")
    worst = getattr(mod, "WORST", None) if mod else None
    if worst:
        terminalreporter.write_line("worst normalised error per check: " + ", ".join(
            f"{k} {v:.3e}" for k, v in sorted(worst.items())))
