"""MI355X-native grouped adapter execution (ACE, arXiv 2609.06072).

Submodules:
  ace        -- ctypes binding of the C-ABI library ``libace.so`` (loads it on import)
  workloads  -- seeded synthetic MoE routing and tensor generators
  build      -- compiles the HIP sources for gfx950

Importing the package itself loads nothing, so the generators work on a host
without a GPU; ``paper_2609_06072_amd.ace`` raises if the library is missing.
"""

__all__ = ["ace", "workloads", "build"]
