"""MI355X-native (gfx950) hot path of Dependency-Aware Revocable Decoding.

The compute lives in ``libdard.so`` (HIP kernels behind a C ABI declared in
``include/dard.h``); :mod:`paper_2608_26574_amd.dard` is a thin ctypes binding
with the same entry-point names.  Importing the package loads nothing; the
library is loaded on first use and its absence is an error.
"""
__all__ = ["dard", "synth"]
