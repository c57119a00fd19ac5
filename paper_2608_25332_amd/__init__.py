"""MI355X-native (gfx950) implementation of ProViP's pruning hot path.

The compute lives in ``libprovip.so`` (hand-written HIP kernels behind a
C ABI, declared in ``include/provip.h``).  ``paper_2608_25332_amd.provip``
is the thin ctypes binding; ``workloads`` draws the seeded synthetic inputs.
Importing the package does not load the GPU library.
"""

__all__ = ["workloads", "provip"]
