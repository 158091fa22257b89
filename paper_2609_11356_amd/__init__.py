"""Descriptor-ordered bf16 GEMM and row reduction for MI355X (gfx950).

The floating-point reduction order of every output is fixed by a descriptor
(group width, K tile, split-K cut points, tile and split combines, partial and
merge precision, FMA fusion, rounding points), never by the tile shape or grid
chosen for speed.  The compute path is the C-ABI library ``libdg.so`` (HIP
kernels for gfx950); :mod:`.dg` is its thin ctypes binding.
"""
__all__ = ["dg", "inputs"]
