"""GCPSL hot path on MI355X (gfx950): HIP kernels behind a C ABI.

Submodules:
  gcpsl   ctypes binding of libgcpsl.so (include/gcpsl.h)
  driver  Alg. 2 loop over the binding (sample -> step -> periodic fuse)
  build   hipcc build of libgcpsl.so
"""
