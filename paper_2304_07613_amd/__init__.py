"""MI355X-native n:m:g sparse weights: compress (magnitude sparsifier) and
sparse x dense product, after STen (arXiv 2304.07613), Section 5.

The compute lives in ``libnmg.so`` (HIP kernels for gfx950 behind a C ABI,
declared in ``include/nmg.h``); :mod:`.nmg` is a thin ctypes binding that only
marshals arguments.  Import the binding explicitly::

    from paper_2304_07613_amd import nmg
"""
__all__ = ["nmg", "synth"]
