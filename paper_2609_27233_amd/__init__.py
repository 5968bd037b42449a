"""Span-merging (UMIM) inference hot path on AMD Instinct MI355X (gfx950).

Submodules:
  lib       ctypes binding of libspanmerge.so (the C ABI in include/spanmerge.h)
  workload  seeded synthetic inputs for the five benchmark workloads
  build     compiles the HIP sources

Importing the package loads nothing; ``lib.load()`` loads the HIP library
and raises if it has not been built.
"""

__all__ = ["lib", "workload", "build"]
