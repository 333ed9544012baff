"""MicroMix hot path for AMD Instinct MI355X (gfx950).

Fused reorder-and-quantize of bf16 activations into MXFP4 / MXFP6 / MXFP8
partitions and a mixed-precision block-scaled GEMM with bf16 output, as HIP
kernels behind a C ABI (include/micromix.h).

Submodules (imported explicitly, so that importing the package loads nothing):
  binding    ctypes layer over libmicromix.so; it fails loudly on import if the
             library is missing
  workloads  seeded synthetic inputs shaped like the paper's layers
  build_lib  hipcc build of libmicromix.so
"""
