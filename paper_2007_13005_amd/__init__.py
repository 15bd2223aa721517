"""smol-mi355x: fused image preprocessing on MI355X (gfx950).

The product is the C-ABI library ``libsmol.so`` built from ``csrc/``; the
Python module ``paper_2007_13005_amd.smol`` is a thin ctypes binding over it.
Importing this package loads nothing; the binding loads the library on first
use and raises if it is missing.
"""
