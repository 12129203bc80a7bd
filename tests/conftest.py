import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter):
    from parity_report import LINES
    if LINES:
        terminalreporter.write_sep("-", "errors against the fp64 oracle")
        for line in LINES:
            terminalreporter.write_line(line)
