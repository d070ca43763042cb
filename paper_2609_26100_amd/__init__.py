"""TSS sparse-depth target verification on MI355X (gfx950).

The product is libtss.so (C ABI in include/tss.h); ``tss`` is its thin ctypes
binding and ``verifier.Verifier`` binds it to torch-owned device buffers.
"""
from . import tss  # noqa: F401
