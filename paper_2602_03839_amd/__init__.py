"""MI355X (gfx950) PULSE patch codec: BF16 sparse-patch encode/apply and
error-feedback sparsification, as hand-written HIP kernels behind a C ABI.

Submodules:
  pulse      ctypes binding to libpulse.so (the C ABI in include/pulse.h)
  workloads  seeded synthetic inputs and parameter-set shapes
"""
__all__ = ["pulse", "workloads"]
