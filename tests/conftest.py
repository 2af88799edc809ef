import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_terminal_summary(terminalreporter):
    """Print the parity lines the GPU tests reported (tests.gpu_helpers.report)."""
    from tests import gpu_helpers
    if gpu_helpers.SUMMARY:
        terminalreporter.section("parity and timing summary")
        for line in gpu_helpers.SUMMARY:
            terminalreporter.write_line(line)
