"""ETA (Elastic Threshold Attention) decode path for AMD Instinct MI355X (gfx950).

The compute lives in ``libeta.so`` (hand-written HIP, C ABI in include/eta.h);
``paper_2609_20888_amd.eta`` is its ctypes binding.  Importing this package
loads nothing; the library is loaded on first use.
"""
__all__ = ["eta"]
