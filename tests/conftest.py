import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    # GPU tests fail (they are never skipped) when no device is present:
    # deselect them with -m "not gpu" on a CPU-only machine.
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library)")
