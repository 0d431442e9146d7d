"""MomentKV hot path on MI355X (gfx950): compress + corrected decode as HIP kernels.

The kernels live in ``libmomentkv.so`` (built from ``csrc/``) behind the C ABI declared
in ``include/momentkv.h``; ``momentkv`` is a thin ctypes binding over it.  Importing
this package does not load the library; the first call does, and raises if the
library is missing.
"""
__version__ = "0.1.0"
