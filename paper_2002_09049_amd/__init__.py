"""MI355X (gfx950) multipoint post-training quantization: the greedy
per-channel fit, its output error and the reconstruction, as hand-written HIP
kernels behind a C ABI (include/mpq.h).

Submodules:
  mpq        Python binding of libmpq.so (imports torch, loads the library)
  workloads  seeded synthetic layer stacks (no arithmetic of the method)
  build      compiles libmpq.so for gfx950
"""
__all__ = ["mpq", "workloads", "build"]
