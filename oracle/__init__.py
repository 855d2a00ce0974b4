"""fp64 CPU oracle of the MoE-layer forward.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the package smoke check and
the benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP kernels.  Every function is pinned by the ``-m "not gpu"`` tests in
``tests/test_oracle_pins.py`` (closed forms, brute force, identities).
"""
from .moe_oracle import *  # noqa: F401,F403
from .moe_oracle import GATE_SIGMOID, GATE_SOFTMAX  # noqa: F401
from . import moe_backward  # noqa: F401,E402
