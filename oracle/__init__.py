"""CPU oracle of the P4Q hot path -- test infrastructure only.

Used by tests/, the smoke check and the benchmark's CPU-baseline leg; never by
the product path.  See p4q_oracle for the definitions it follows.
"""
from .p4q_oracle import *  # noqa: F401,F403
from . import p4q_oracle  # noqa: F401
