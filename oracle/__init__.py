"""CPU oracle of the MoE-layer hot path (test infrastructure only).

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this package.
"""
from .moe_oracle import *  # noqa: F401,F403
from . import moe_oracle  # noqa: F401
