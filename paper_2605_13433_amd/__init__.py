"""MI355X (gfx950) jagged HSTU attention: C-ABI HIP library + thin binding.

Submodules:
  hstu    ctypes binding of include/hstu_jagged.h (loads libhstu_jagged.so)
  inputs  seeded synthetic workloads (no attention arithmetic)
  build   compiles the HIP library in-tree
"""
__all__ = ["hstu", "inputs", "build"]
