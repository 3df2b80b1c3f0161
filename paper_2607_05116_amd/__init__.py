"""MI355X-native hot path of CAP's expert-parallel MoE layer (HIP for gfx950).

The compute lives in libcap.so (C ABI in include/cap.h).  Submodules:
  capi      ctypes binding with the C function names
  layer     device buffers and the chained calls of one layer step
  placement co-activation placement (Algorithm 1 + node stage) on the host
  build     hipcc build of libcap.so
Importing the package itself loads nothing; `capi` fails loudly when the
library is missing.
"""
