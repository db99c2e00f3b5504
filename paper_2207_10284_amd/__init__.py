"""MRA-2 multiresolution approximate self-attention for AMD Instinct MI355X (gfx950).

The compute path is the C-ABI library ``libmra.so`` (hand-written HIP kernels);
``ops`` is its thin Python binding. Importing the package loads nothing; the
library is opened on first use and a missing build raises at that point.
"""
__all__ = ["ops", "inputs"]
