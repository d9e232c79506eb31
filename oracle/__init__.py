"""CPU oracle for the per-micro-step MoE expert layer (test infrastructure).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. The product path (the HIP library and its binding)
never calls it and shares no code with it.
"""
from . import foremoe_oracle  # noqa: F401
from . import foremoe_transfer  # noqa: F401
from .foremoe_oracle import *  # noqa: F401,F403
