import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Print the figures the parity tests recorded (near-ties at kept-set
    boundaries, worst error-to-bound ratios), which pytest would otherwise
    drop with the captured output of passing tests."""
    from tests.parity import REPORT
    if not REPORT:
        return
    terminalreporter.write_sep("-", "parity report")
    for key in sorted(REPORT):
        terminalreporter.write_line(f"{key}: {REPORT[key]}")
