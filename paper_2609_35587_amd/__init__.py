"""Batched hardware-aware candidate scoring on MI355X (gfx950).

The scored path lives in ``libhwsel.so`` (HIP kernels behind a C ABI, see
``include/hwsel.h``); ``paper_2609_35587_amd.hwsel`` is its ctypes binding.
"""
