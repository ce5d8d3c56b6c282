"""MI355X-native R-iKFAD optimiser step (Rank-1 iKFAD, Rajpal & Leimkuhler).

The step runs in hand-written HIP kernels for gfx950 behind the C ABI
declared in ``include/rikfad.h``; :mod:`paper_2609_30342_amd.rikfad` is the
thin ctypes binding with the same entry-point names.  Importing the package
loads nothing; the native library is opened on first use and its absence is
an error (there is no CPU fallback).
"""
__all__ = ["rikfad", "synth"]
