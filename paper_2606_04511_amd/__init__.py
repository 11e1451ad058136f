"""MI355X (gfx950) implementation of SparDA's selection + block-sparse attention hot path.

Submodules:
  sparda  -- ctypes binding of libsparda.so (C ABI in include/sparda.h)
  build   -- hipcc build of libsparda.so
  inputs  -- seeded synthetic workloads (random draws and layout only)
"""
