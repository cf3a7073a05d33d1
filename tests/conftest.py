import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an AMD GPU (gfx950) and the built HIP library")


def pytest_terminal_summary(terminalreporter):
    """Prints the parity records the GPU tests collected (selection tie rows and swaps, error
    statistics), so that they are part of the run's output even when every test passes."""
    parity = sys.modules.get("tests._parity")
    lines = getattr(parity, "REPORTS", None) if parity else None
    if lines:
        terminalreporter.section("parity records")
        for line in lines:
            terminalreporter.write_line(line)
