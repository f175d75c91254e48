"""WnW (Waxing-and-Waning KV cache) per-token decode step on MI355X (gfx950).

The compute path is the HIP library ``libwnw.so`` (C ABI in ``include/wnw.h``); ``wnw`` is its
ctypes binding.  Importing ``paper_2608_22704_amd.wnw`` fails loudly when the library is not
built: there is no CPU fallback.
"""
__all__ = ["wnw", "build"]
