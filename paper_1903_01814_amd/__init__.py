"""MI355X-native hexagonal convolution and pooling (HexagDLy, arXiv:1903.01814).

The compute lives in libhexconv.so (HIP kernels for gfx950, C ABI declared in
include/hexconv.h); ``hexconv`` is its Python binding, ``nn`` puts it behind
torch autograd as layers (HexConv2d, HexMaxPool2d, HexAvgPool2d), and
``inputs`` is the seeded synthetic workload generator.
"""
