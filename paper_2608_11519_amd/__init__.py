"""FLARE++ mixer forward on AMD MI355X (gfx950).

The compute path is the C-ABI library ``libflarepp.so`` (hand-written HIP
kernels); :mod:`paper_2608_11519_amd.flarepp` is the thin Python binding over
it.  Importing this package loads nothing; the binding loads the library on
first use and raises if it is missing.
"""

__all__ = ["inputs", "flarepp"]
