"""MI355X (gfx950) summed-area-table box-convolution layer.

The compute path is the HIP library ``libboxconv.so`` (C ABI declared in
``include/boxconv.h``); :mod:`paper_1906_11367_amd.boxconv` is a thin ctypes
binding with the same entry-point names.  The library is loaded lazily, on
first use, and a missing library is an error: there is no fallback path.
"""
__all__ = ["workloads"]
