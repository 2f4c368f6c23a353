"""CPU fp64 oracle for the FAL / FAL+ / GPT training step.

Test infrastructure: imported only by tests/, the smoke check and the
benchmark's CPU-baseline leg.  Never used by the product path.
"""
from .fal_oracle import *  # noqa: F401,F403
