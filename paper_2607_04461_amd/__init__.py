"""MI355X-native batched draft generation for Flash-BoN (arXiv 2607.04461).

``flashbon``: ctypes binding of libflashbon.so (the C ABI); ``pool``: a candidate pool driven through
it; ``synth``: seeded synthetic inputs; ``build``: hipcc build of the library for gfx950.
"""
