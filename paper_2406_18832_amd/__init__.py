"""OutlierTune's per-channel-quantized linear on MI355X (gfx950).

The compute lives in ``libot.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/ot.h``); :mod:`paper_2406_18832_amd.ot` is the thin
Python binding with the same entry-point names.  Importing this package does
not load the library; ``ot`` loads it on first use and raises if it is
missing.
"""
__all__ = ["ot", "synth"]
