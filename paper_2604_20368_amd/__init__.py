"""MI355X (gfx950) Nystrom-approximated Laplacian-kernel attention.

The compute lives in the HIP library ``liblapattn.so`` (C ABI in
``include/lapattn.h``); :mod:`paper_2604_20368_amd.lapattn` is the thin ctypes
binding with the same entry-point names.  Importing this package loads nothing;
the library is opened on first use and its absence is an error (there is no
CPU fallback).
"""
__all__ = ["lapattn"]
