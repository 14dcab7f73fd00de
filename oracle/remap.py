"""Oracle: layout remap, a pure permutation of elements.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

For every logical index x of the common logical view, the element stored at
``L_src.apply(x)`` in the source buffer is copied to ``L_dst.apply(x)`` in the
destination buffer.  This is the data-movement meaning of a layout pair in
Section III (a layout maps a logical index to its physical position); the 2D
transpose of Section V-C (Table V) is the case L_src = Row, L_dst = Col.
"""
from __future__ import annotations

import numpy as np

from .layout import ExpandBy, canon_unflatten, prod


def phys_size(layout):
    """Number of physical positions of a layout: the original extents of an
    ExpandBy (Figure 9), the logical size otherwise."""
    return prod(layout.n) if isinstance(layout, ExpandBy) else prod(layout.dims())


def remap(src_layout, dst_layout, src, chunk=1 << 22, fill=0):
    """Return dst with dst[L_dst.apply(x)] = src[L_src.apply(x)] for all x.

    ``src`` is a flat numpy array of any dtype with phys_size(L_src) elements;
    dst has phys_size(L_dst) elements.  Under ExpandBy, apply gives -1 for a
    point outside the original extents (Section III-D): such a point is not
    written when it is the destination's, and writes ``fill`` when it is only
    the source's (padding).  The logical index space is walked in chunks only
    to bound memory."""
    dims = list(src_layout.dims())
    if list(dst_layout.dims()) != dims:
        raise ValueError("layouts have different logical shapes")
    n = prod(dims)
    src = np.asarray(src).reshape(-1)
    if src.size != phys_size(src_layout):
        raise ValueError("source size does not match the layout")
    nd = phys_size(dst_layout)
    dst = np.full(nd, fill, dtype=src.dtype)
    written = np.zeros(nd, dtype=bool)
    for lo in range(0, n, chunk):
        x = np.arange(lo, min(n, lo + chunk), dtype=np.int64)
        coords = canon_unflatten(dims, x)
        s = np.asarray(src_layout.apply(coords), dtype=np.int64)
        d = np.asarray(dst_layout.apply(coords), dtype=np.int64)
        keep = d >= 0
        s, d = s[keep], d[keep]
        if written[d].any():
            raise ValueError("destination position written twice")
        has = s >= 0
        dst[d[has]] = src[s[has]]
        written[d] = True
    if not written.all():
        raise ValueError("destination layout is not onto: some positions never written")
    return dst
