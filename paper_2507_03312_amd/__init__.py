"""MI355X (gfx950) hot path of MPX's mixed-precision training step.

``binding``  ctypes binding of libmpx.so (the C ABI in include/mpx.h)
``train``    the training step (MLP / ViT) composed from libmpx calls
``sweep``    the standalone optimizer sweep over a list of gradient tensors
``build``    compiles libmpx.so with hipcc for gfx950

Importing ``binding`` (and the modules that use it) requires the built
library; there is no fallback implementation.
"""
