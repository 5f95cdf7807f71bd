import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Counts that parity tests record while they run (near-threshold exclusions, kept-list
# disagreements, gradient error ratios); printed in the terminal summary, which pytest
# shows even with -q, so the run's record holds them.
RECORDS = []


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    if not RECORDS:
        return
    terminalreporter.section("parity counts")
    for line in RECORDS:
        terminalreporter.write_line(line)
