"""MI355X-native hexagonal convolution and pooling (HexagDLy, arXiv:1903.01814).

The compute lives in libhexconv.so (HIP kernels for gfx950, C ABI declared in
include/hexconv.h); ``hexconv`` is its Python binding and ``inputs`` the
seeded synthetic workload generator.
"""
