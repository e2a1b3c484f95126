"""fp64 CPU oracle of the MoE-layer hot path (test infrastructure only).

Importable only by the test suite, the smoke check and the CPU-baseline leg of
the benchmark.  Nothing in the HIP library or its Python binding imports it.
"""
from .moe_oracle import *  # noqa: F401,F403
from .moe_oracle import MergePlan, SlotWeights  # noqa: F401
