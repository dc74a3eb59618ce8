import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: runs HIP kernels through the C-ABI library (needs an MI355X)")
    config.addinivalue_line(
        "markers", "slow: CPU test that takes more than a few seconds")
