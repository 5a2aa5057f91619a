"""MI355X-native hot path of SparseSpec-L's self-speculative decode step.

Submodules:
  workloads  seeded synthetic inputs (no method arithmetic)
  binding    ctypes binding of the C-ABI library (loaded on first use)
"""
