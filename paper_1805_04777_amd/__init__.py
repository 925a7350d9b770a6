"""ConvCRF mean-field inference on AMD Instinct MI355X (gfx950).

The compute path is the C-ABI library ``libconvcrf.so`` (hand-written HIP
kernels, declared in ``include/convcrf.h``); :mod:`.convcrf` is a thin ctypes
binding over it, and :mod:`.synth` generates seeded synthetic workloads.
Importing the package loads nothing; the library is loaded on first use and
a missing library is an error, never a fallback.
"""
__all__ = ["convcrf", "synth"]
