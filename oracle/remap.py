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

from .layout import canon_unflatten, prod


def remap(src_layout, dst_layout, src, chunk=1 << 22):
    """Return dst with dst[L_dst.apply(x)] = src[L_src.apply(x)] for all x.

    ``src`` is a flat numpy array of any dtype with prod(dims) elements.  The
    logical index space is walked in chunks only to bound memory."""
    dims = list(src_layout.dims())
    if list(dst_layout.dims()) != dims:
        raise ValueError("layouts have different logical shapes")
    n = prod(dims)
    src = np.asarray(src).reshape(-1)
    if src.size != n:
        raise ValueError("source size does not match the layout")
    dst = np.empty_like(src)
    written = np.zeros(n, dtype=bool)
    for lo in range(0, n, chunk):
        x = np.arange(lo, min(n, lo + chunk), dtype=np.int64)
        coords = canon_unflatten(dims, x)
        s = np.asarray(src_layout.apply(coords), dtype=np.int64)
        d = np.asarray(dst_layout.apply(coords), dtype=np.int64)
        dst[d] = src[s]
        written[d] = True
    if not written.all():
        raise ValueError("destination layout is not onto: some positions never written")
    return dst
