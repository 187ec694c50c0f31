"""MI355X-native hot path of thought-level beam search (population decode).

The product is libgambit.so (HIP kernels for gfx950 behind the C ABI in
include/gambit.h); ``gambit`` is its ctypes binding and ``runner`` drives a
synthetic population workload through it.
"""
