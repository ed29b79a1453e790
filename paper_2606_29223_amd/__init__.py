"""MI355X (gfx950) implementation of the Depth Exploration Decoding step.

The decode path lives in libdex.so (HIP kernels + host engine, C ABI in
include/dex.h); `dexlib` is its ctypes binding.
"""
