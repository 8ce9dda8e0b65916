"""MI355X (gfx950) implementation of the scalable-Shampoo hot path.

The computation lives in libshampoo.so (hand-written HIP, C ABI in
include/shampoo.h); ``binding`` is its thin ctypes binding.
"""
