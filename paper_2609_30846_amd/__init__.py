"""ipk: integer-only relative-position multi-head self-attention on MI355X (gfx950).

The block of Sec. 3.1 of the I-Parakeet paper, as hand-written HIP kernels behind
the C ABI declared in include/ipk.h.  ``ipk`` is the ctypes binding of that ABI;
``build`` compiles ``libipk.so`` with hipcc.
"""

from . import ipk  # noqa: F401

__all__ = ["ipk"]
