"""Oracle: dense GEMM with operands read through layouts, in fp64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

C[m, n] = sum_k A[m, k] * B[k, n] (the matrix product of Section II and
Section V-A), where the logical element A[m, k] is the fp16/bf16 value stored at
``L_A.apply(m, k)`` of A's buffer, likewise for B, and C is written at
``L_C.apply(m, n)``.  Inputs are decoded exactly to fp64; every product of two
fp16 or bf16 values is exact in fp64, and the fp64 sum over K <= 8192 is within
about 1e-12 relative of the real-number result, so the summation order does not
matter at the tolerances used against fp32-accumulating kernels.
"""
from __future__ import annotations

import numpy as np

from .layout import canon_unflatten, prod


def decode(buf, dtype):
    """Exact decode of a flat buffer of 'f16', 'bf16' (given as uint16 bits or
    float16) or 'f32' values to fp64."""
    a = np.asarray(buf).reshape(-1)
    if dtype == "f16":
        return a.view(np.float16).astype(np.float64) if a.dtype != np.float16 else a.astype(np.float64)
    if dtype == "bf16":
        bits = a.view(np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return a.view(np.float32).astype(np.float64)
    raise ValueError(dtype)


def logical_matrix(buf, layout, dtype, rows=None):
    """The logical 2D matrix held by ``buf`` in ``layout``, decoded to fp64.

    ``rows`` optionally selects a subset of logical rows."""
    d0, d1 = layout.dims()
    vals = decode(buf, dtype)
    r = np.arange(d0, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    rr = np.repeat(r, d1)
    cc = np.tile(np.arange(d1, dtype=np.int64), r.size)
    pos = np.asarray(layout.apply([rr, cc]), dtype=np.int64)
    return vals[pos].reshape(r.size, d1)


def gemm(a_buf, b_buf, la, lb, dtype, rows=None):
    """fp64 logical product R = A @ B (rows of R optionally subsampled).

    Returns R as a logical [M or len(rows), N] fp64 matrix."""
    m, k = la.dims()
    k2, n = lb.dims()
    if k != k2:
        raise ValueError("inner dimensions differ")
    a = logical_matrix(a_buf, la, dtype, rows)
    b = logical_matrix(b_buf, lb, dtype)
    return a @ b


def store(r, lc, rows=None):
    """Place the logical result R into a flat fp64 buffer in layout L_C (only
    when all rows are present)."""
    m, n = lc.dims()
    assert rows is None and r.shape == (m, n)
    out = np.empty(m * n, dtype=np.float64)
    x = np.arange(m * n, dtype=np.int64)
    coords = canon_unflatten([m, n], x)
    out[np.asarray(lc.apply(coords), dtype=np.int64)] = r.reshape(-1)
    return out


def check_tolerance(c, r, max_rel=2e-2, fro_rel=1e-3):
    """Error of a computed logical result c against the fp64 oracle r.

    Per element: |c - r| / max(|r|, ||r||_F / sqrt(#elements)) <= max_rel; and
    ||c - r||_F / ||r||_F <= fro_rel.  Returns (ok, max_rel_err, fro_rel_err)."""
    c = np.asarray(c, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    fro = np.linalg.norm(r)
    floor = fro / np.sqrt(r.size) if r.size else 0.0
    denom = np.maximum(np.abs(r), floor)
    denom = np.where(denom == 0, 1.0, denom)
    err = np.abs(c - r)
    mre = float((err / denom).max()) if r.size else 0.0
    fre = float(np.linalg.norm(c - r) / fro) if fro > 0 else float(np.linalg.norm(c - r))
    return (mre <= max_rel and fre <= fro_rel), mre, fre


def n_elems(layout):
    return prod(layout.dims())
