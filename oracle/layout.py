"""Oracle: the LEGO layout algebra, evaluated point by point.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Follows Section III-B of the paper: the grammar of Figure 3, the apply/inv/dims
semantics of RegP, GenP and OrderBy in Figure 4 and of GroupBy in Figure 5, the
dot notation of Equation (2) and the syntactic sugar (Row, Col, TileBy,
TileOrderBy) defined right after it; ExpandBy follows Figure 9 (Section III-D).

Every function works on Python ints and, elementwise, on numpy int64 arrays, so
one definition serves single points and whole index spaces.

Readings of passages that are ambiguous or garbled (each one is pinned by a
test in ``tests/test_oracle_pins.py``):

* Chain order.  In dot notation ``GroupBy(g).OrderBy(O_a).OrderBy(O_b)`` the
  reorderings are applied left to right by ``apply`` (O_a first).  Figure 5
  iterates ``reverse`` of the grammar's list, so the grammar form lists them in
  the opposite order.  Pinned by the Figure 6 walk-through ([4,2] -> 23 -> 15).
* sigma is a gather: ``sigma(v)_k = v[sigma_k]`` (1-based).  Pinned by Figure 6
  and the printed sigma_{2x3}, sigma_{3x2}.
* Col([n_1..n_d]) keeps the logical dims [n_1..n_d] and makes the first index
  fastest: ``RegP([n_1..n_d], [d..1])``.  The printed form reverses the dims as
  well, which is not column-major for non-square shapes; the usage "B is
  Col(K,N)" in Section V-A needs the column-major meaning.
* TileOrderBy_{q x d}(P^1..P^q) over full dims N_k = prod_h n^h_k is
  ``GroupBy(N).OrderBy(RegP(I, sigma_{d x q}^{-1})).OrderBy(P^1, .., P^q)``
  with I = sigma_{d x q}(tile-major dims) the interleaved digit dims: full
  coordinates go to tile-major storage, level h ordered by P^h.  The printed
  definition is garbled.
* Figure 2's p^{-1} (not shown in the paper) is B^{-1}([n1,n2], n1*n2-1-x).
* The antidiagonal order of Figure 7 is taken from what it computes: the
  antidiagonals in turn, rows increasing within one (the printed code's real
  division and square root are not needed to count that way).
* Morton (Z) order puts column bits at even and row bits at odd positions, so
  every 2x2 block reads 0,1,2,3 in row-major order.
* The XOR swizzle over [R, C] with vector width v and row divisor s is
  ``r*C + ((c/v) ^ ((r/s) % (C/v)))*v + c%v`` (C/v a power of two).
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "canon_flatten", "canon_unflatten", "sigma_gather", "sigma_inverse",
    "sigma_dq", "RegP", "GenP", "OrderBy", "GroupBy", "ExpandBy", "Row", "Col",
    "TileBy", "TileOrderBy", "reverse_genp", "antidiag", "antidiag_inv",
    "antidiag_genp", "morton", "morton_inv", "morton_genp", "xor_swizzle",
    "xor_swizzle_inv", "xor_swizzle_genp", "as_layout", "prod",
]


def prod(xs):
    p = 1
    for x in xs:
        p *= int(x)
    return p


# ---------------------------------------------------------------- Figure 4 --
def canon_flatten(n, idx):
    """Canonical bijection B_n (Figure 4): Horner flattening, last dim fastest."""
    assert len(n) == len(idx)
    f = 0
    for nk, ik in zip(n, idx):
        f = f * int(nk) + ik
    return f


def canon_unflatten(n, x):
    """Inverse canonical bijection B^{-1}_n (Figure 4): repeated div/mod, last dim
    fastest.  Returns a list of len(n) coordinates."""
    out = [None] * len(n)
    for k in range(len(n) - 1, 0, -1):
        out[k] = x % int(n[k])
        x = x // int(n[k])
    out[0] = x
    return out


def sigma_gather(sigma, v):
    """Apply a constant permutation of dimensions as a gather (Figure 4, RegP):
    ``sigma(v)_k = v[sigma_k]`` with 1-based sigma."""
    return [v[s - 1] for s in sigma]


def sigma_inverse(sigma):
    """sigma^{-1}: scatter [1..d] at the positions of sigma (Figure 4)."""
    inv = [0] * len(sigma)
    for k, s in enumerate(sigma):
        inv[s - 1] = k + 1
    return inv


def sigma_dq(d, q):
    """sigma_{d x q} = flatten(A), A[k][h] = k+1+d*h (sugar after Equation (2))."""
    return [k + 1 + d * h for k in range(d) for h in range(q)]


# ------------------------------------------------------------ permutations --
class RegP:
    """Regular permutation RegP(tile, sigma) (Figure 3; semantics Figure 4)."""

    def __init__(self, dims, sigma):
        self.n = [int(x) for x in dims]
        self.sigma = [int(s) for s in sigma]
        assert sorted(self.sigma) == list(range(1, len(self.n) + 1)), "sigma not a permutation"

    def dims(self):
        return list(self.n)

    def size(self):
        return prod(self.n)

    def apply(self, idx):
        return canon_flatten(sigma_gather(self.sigma, self.n), sigma_gather(self.sigma, list(idx)))

    def inv(self, x):
        return sigma_gather(sigma_inverse(self.sigma),
                            canon_unflatten(sigma_gather(self.sigma, self.n), x))


class GenP:
    """General (user-defined) permutation GenP(tile, f, f^inv) (Figures 3, 4)."""

    def __init__(self, dims, f, finv, name="genp"):
        self.n = [int(x) for x in dims]
        self.f = f
        self.finv = finv
        self.name = name

    def dims(self):
        return list(self.n)

    def size(self):
        return prod(self.n)

    def apply(self, idx):
        return self.f(*idx)

    def inv(self, x):
        return list(self.finv(x))


class OrderBy:
    """OrderBy(Prm_1 .. Prm_q) (Figure 3; semantics Figure 4)."""

    def __init__(self, *pieces):
        assert pieces, "OrderBy needs at least one permutation"
        self.pieces = list(pieces)

    def dims(self):
        out = []
        for p in self.pieces:
            out += p.dims()
        return out

    def size(self):
        return prod(self.dims())

    def apply(self, idx):
        """Outermost piece first; each step flattens its slice of the index and
        accumulates ``cur + flat * |piece|``."""
        flat = 0
        pos = 0
        for p in self.pieces:
            d = len(p.dims())
            cur = p.apply(idx[pos:pos + d])
            flat = cur + flat * p.size()
            pos += d
        assert pos == len(idx)
        return flat

    def inv(self, x):
        """Innermost piece first: peel ``x % |piece|``, invert it, prepend."""
        out = []
        for p in reversed(self.pieces):
            sz = p.size()
            cur = x % sz
            x = x // sz
            out = list(p.inv(cur)) + out
        return out


class GroupBy:
    """GroupBy(tiles, OrderBy chain) (Figure 3; semantics Figure 5).

    ``GroupBy(t1, t2, ...)`` takes the tile levels of the logical view (their
    concatenation is the logical index); ``.OrderBy(...)`` appends a reordering
    in dot notation (Equation (2)), which is also application order."""

    def __init__(self, *tiles, chain=()):
        self.tiles = [list(map(int, t)) for t in tiles]
        self.chain = list(chain)
        n = prod(self.dims())
        for o in self.chain:
            if o.size() != n:
                raise ValueError("GroupBy and OrderBy element counts differ")

    def OrderBy(self, *pieces):  # noqa: N802  (paper notation)
        return GroupBy(*self.tiles, chain=self.chain + [OrderBy(*pieces)])

    def dims(self):
        out = []
        for t in self.tiles:
            out += t
        return out

    def size(self):
        return prod(self.dims())

    def apply(self, idx):
        """Figure 5 apply: flatten in the logical view, then for each reorder O
        (dot order) unflatten over O.dims and apply O."""
        flat = canon_flatten(self.dims(), list(idx))
        for o in self.chain:
            flat = o.apply(canon_unflatten(o.dims(), flat))
        return flat

    def inv(self, x):
        """Figure 5 inv: for each reorder in reverse dot order apply O.inv and
        flatten over O.dims; finally unflatten in the logical view."""
        for o in reversed(self.chain):
            x = canon_flatten(o.dims(), o.inv(x))
        return canon_unflatten(self.dims(), x)


class ExpandBy:
    """ExpandBy(n, n', G) for partial tiles (Figure 9, Section III-D).

    apply returns -1 for points of the expanded space outside n."""

    def __init__(self, n, n_exp, g):
        self.n = list(map(int, n))
        self.ne = list(map(int, n_exp))
        self.g = g

    def dims(self):
        return self.g.dims()

    def apply(self, idx):
        flat = self.g.apply(idx)
        ip = canon_unflatten(self.ne, flat)
        inside = True
        for a, b in zip(ip, self.n):
            inside = inside & (a < b)
        f = canon_flatten(self.n, ip)
        return np.where(inside, f, -1) if isinstance(inside, np.ndarray) else (f if inside else -1)

    def inv(self, x):
        i = canon_unflatten(self.n, x)
        return self.g.inv(canon_flatten(self.ne, i))


# ------------------------------------------------------------------- sugar --
def Row(*n):  # noqa: N802
    """Row([n_1..n_d]) = RegP(n, [1..d])."""
    n = _dims_arg(n)
    return RegP(n, list(range(1, len(n) + 1)))


def Col(*n):  # noqa: N802
    """Col([n_1..n_d]) = RegP([n_1..n_d], [d..1]) (reading: first index fastest)."""
    n = _dims_arg(n)
    return RegP(n, list(range(len(n), 0, -1)))


def TileBy(*tiles):  # noqa: N802
    """TileBy_{q x d}(T^1..T^q) = GroupBy(T^1..T^q).OrderBy(RegP(T^1..T^q, sigma_{d x q}))."""
    q = len(tiles)
    d = len(tiles[0])
    cat = [int(x) for t in tiles for x in t]
    return GroupBy(*tiles).OrderBy(RegP(cat, sigma_dq(d, q)))


def TileOrderBy(*pieces):  # noqa: N802
    """TileOrderBy_{q x d}(P^1..P^q) (reading in the module docstring)."""
    q = len(pieces)
    d = len(pieces[0].dims())
    tile_major = [int(x) for p in pieces for x in p.dims()]
    s = sigma_dq(d, q)
    interleaved = sigma_gather(s, tile_major)
    full = [prod(p.dims()[k] for p in pieces) for k in range(d)]
    return GroupBy(full).OrderBy(RegP(interleaved, sigma_inverse(s))).OrderBy(*pieces)


def as_layout(piece):
    """A single permutation used as a whole layout: GroupBy(dims).OrderBy(piece)."""
    return GroupBy(piece.dims()).OrderBy(piece)


def _dims_arg(n):
    if len(n) == 1 and isinstance(n[0], (list, tuple)):
        return [int(x) for x in n[0]]
    return [int(x) for x in n]


# ---------------------------------------------------- named permutations --
def reverse_genp(n1, n2):
    """Figure 2's per-tile permutation p(i,j) = (n1-1-i)*n2 + (n2-1-j) and its
    inverse (reading: B^{-1}([n1,n2], n1*n2-1-x))."""
    def f(i, j):
        return (n1 - 1 - i) * n2 + (n2 - 1 - j)

    def finv(x):
        return canon_unflatten([n1, n2], n1 * n2 - 1 - x)

    return GenP([n1, n2], f, finv, name="reverse")


def _antidiag_starts(n):
    """start[d] for d = 0..2n-1: the number of points on the antidiagonals
    before antidiagonal d of an n x n tile (antidiagonal d, i + j = d, holds
    min(d + 1, 2n - 1 - d) points)."""
    d = np.arange(2 * n - 1, dtype=np.int64)
    return np.concatenate([[0], np.cumsum(np.minimum(d + 1, 2 * n - 1 - d))])


def antidiag(n, i, j):
    """Antidiagonal order of an n x n tile (Figure 7): the elements are
    numbered antidiagonal by antidiagonal (i + j ascending) and, within one,
    by increasing row.  The number of (i, j) is the count of the points on the
    earlier antidiagonals plus the points of its own antidiagonal with a
    smaller row (the rows of antidiagonal d start at max(0, d - n + 1))."""
    d = np.asarray(i) + np.asarray(j)
    return _antidiag_starts(n)[d] + i - np.maximum(0, d - n + 1)


def antidiag_inv(n, x):
    """Inverse of :func:`antidiag`: the antidiagonal whose block of numbers
    holds x (a search in the cumulative counts), then the row from the offset
    of x within it."""
    start = _antidiag_starts(n)
    d = np.searchsorted(start, x, side="right") - 1
    i = x - start[d] + np.maximum(0, d - n + 1)
    return [i, d - i]


def antidiag_genp(n):
    return GenP([n, n], lambda i, j: antidiag(n, i, j), lambda x: antidiag_inv(n, x),
                name="antidiag")


def _bits(v):
    return max(0, (int(v) - 1).bit_length())


def morton(nbits_r, nbits_c, i, j):
    """Morton (Z) order over [2^nbits_r, 2^nbits_c]: bits of the column index at
    even and of the row index at odd positions while both remain, then the
    remaining bits of the longer coordinate on top."""
    z = 0
    pos = 0
    for b in range(max(nbits_r, nbits_c)):
        if b < nbits_c:
            z = z + ((j >> b) & 1) * (1 << pos)
            pos += 1
        if b < nbits_r:
            z = z + ((i >> b) & 1) * (1 << pos)
            pos += 1
    return z


def morton_inv(nbits_r, nbits_c, z):
    i = 0
    j = 0
    pos = 0
    for b in range(max(nbits_r, nbits_c)):
        if b < nbits_c:
            j = j + ((z >> pos) & 1) * (1 << b)
            pos += 1
        if b < nbits_r:
            i = i + ((z >> pos) & 1) * (1 << b)
            pos += 1
    return [i, j]


def morton_genp(n1, n2):
    br, bc = _bits(n1), _bits(n2)
    assert (1 << br) == n1 and (1 << bc) == n2, "Morton needs power-of-two sides"
    return GenP([n1, n2], lambda i, j: morton(br, bc, i, j),
                lambda z: morton_inv(br, bc, z), name="morton")


def xor_swizzle(R, C, v, s, r, c):  # noqa: N803
    """XOR swizzle over [R, C] (reading in the module docstring)."""
    g = C // v
    return r * C + ((c // v) ^ ((r // s) % g)) * v + c % v


def xor_swizzle_inv(R, C, v, s, x):  # noqa: N803
    g = C // v
    r = x // C
    rest = x % C
    c = ((rest // v) ^ ((r // s) % g)) * v + rest % v
    return [r, c]


def xor_swizzle_genp(R, C, v, s):  # noqa: N803
    g = C // v
    assert C % v == 0 and g & (g - 1) == 0, "C/v must be a power of two"
    return GenP([R, C], lambda r, c: xor_swizzle(R, C, v, s, r, c),
                lambda x: xor_swizzle_inv(R, C, v, s, x), name="xor_swizzle")


# ------------------------------------------------------------ enumeration --
def apply_all(layout, dtype=np.int64):
    """apply() on every logical index, in logical row-major order."""
    n = layout.size()
    x = np.arange(n, dtype=np.int64)
    coords = canon_unflatten(layout.dims(), x)
    return np.asarray(layout.apply(coords), dtype=dtype)


def inv_all(layout):
    """inv() on every physical index; returns int64 [N, rank]."""
    n = layout.size()
    x = np.arange(n, dtype=np.int64)
    coords = layout.inv(x)
    return np.stack([np.broadcast_to(np.asarray(c, dtype=np.int64), (n,)) for c in coords], axis=1)
