"""Shared pytest configuration: the ``gpu`` marker and repo-root imports."""
import os
import sys

# a 16-stream pool plus torch's streams need their own HIP hardware queues; set
# before anything in the test process initialises HIP
os.environ.setdefault("GPU_MAX_HW_QUEUES", "24")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU; parity tests through the C-ABI")
