"""Fused scaled-dot-product attention, forward and backward, for MI355X (gfx950).

The compute path is the C-ABI library ``libattn.so`` (hand-written HIP
kernels); ``paper_2608_17379_amd.attn`` is its thin ctypes binding.  Importing
this package loads nothing; the binding loads the library on first use and
raises if it is missing.
"""
