"""MI355X-native forward of one Mixture-of-Experts layer on one expert-parallel rank.

Hand-written HIP kernels for gfx950 behind a C ABI (``include/moe.h``); this
package holds the kernels' sources (``csrc/``), the build step (``build.py``), a
thin ctypes binding (``moe.py``) and the seeded workload generator
(``workloads.py``).  Importing the package loads nothing; ``moe.lib()`` loads the
built library and raises if it is missing.
"""
__all__ = ["workloads"]
