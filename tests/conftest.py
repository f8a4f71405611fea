import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Rows compared with the oracle on each named workload (GPU runs)."""
    mod = sys.modules.get("tests.gpu_harness")
    lines = getattr(mod, "COVERAGE", None) if mod else None
    if lines:
        terminalreporter.section("oracle parity coverage of the named workloads")
        for line in lines:
            terminalreporter.write_line(line)
