"""MI355X-native concurrent independent GEMMs (GOLDYLOC, arXiv 2409.02227).

libgdy.so (built from csrc/) holds the GO-Kernels, the dynamic selector and
the concurrent launcher behind the C-ABI in include/gdy.h; ``gdy`` is its
ctypes binding and ``inputs`` the seeded workload generators.  Importing
this package loads nothing; ``paper_2409_02227_amd.gdy.Context`` loads the
library and raises if it has not been built.
"""
import os

# HIP maps streams onto at most GPU_MAX_HW_QUEUES hardware queues per
# process (4 by default), which would serialise concurrency degrees above 4.
# Only effective if set before the process first initialises HIP.
os.environ.setdefault("GPU_MAX_HW_QUEUES", "24")

__all__ = ["gdy", "inputs", "build"]
