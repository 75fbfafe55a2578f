"""fp64 CPU oracle for ACE grouped adapter execution.

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the bench's
cpu_baseline leg, never by the library or its binding.
"""
from .ace_oracle import *  # noqa: F401,F403
from . import consolidation_oracle  # noqa: F401  (CKA, grouping, consolidated init)
