"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every expected value is printed
in the paper (fixtures under tests/golden/), a closed form derived by hand, a
library routine (numpy) on a special case, or brute force on tiny inputs.
"""
import itertools
import os

import numpy as np
import pytest

from oracle import layout as L
from oracle import remap as R
from oracle import gemm as G

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fig2():
    return L.GroupBy([6, 4], chain=[L.OrderBy(L.RegP([2, 2], [2, 1]), L.reverse_genp(3, 2))])


def _eq2():
    return (L.GroupBy([6, 6])
            .OrderBy(L.RegP([2, 3, 2, 3], [1, 3, 2, 4]))
            .OrderBy(L.RegP([2, 2], [2, 1]), L.antidiag_genp(3)))


def _golden_examples():
    rows = {}
    with open(os.path.join(GOLDEN, "worked_examples.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name, _, inp, exp = [x.strip() for x in line.split("|")]
            rows[name] = (inp, eval(exp))  # fixture values are plain literals
    return rows


EX = _golden_examples()


# ------------------------------------------------------------ worked examples
def test_fig2_worked_example():
    lay = _fig2()
    assert L.canon_flatten([6, 4], [4, 1]) == EX["fig2_logical_flat"][1]
    assert lay.apply([4, 1]) == EX["fig2_apply"][1]
    assert L.canon_unflatten([2, 2, 3, 2], lay.apply([4, 1])) == EX["fig2_apply_digits"][1]
    assert lay.inv(6) == EX["fig2_inv"][1]


def test_fig6_eq2_worked_example():
    o2 = L.GroupBy([6, 6]).OrderBy(L.RegP([2, 3, 2, 3], [1, 3, 2, 4]))
    assert L.canon_flatten([6, 6], [4, 2]) == EX["fig6_logical_flat"][1]
    assert o2.apply([4, 2]) == EX["fig6_after_O2"][1]
    assert L.canon_unflatten([2, 2, 3, 3], o2.apply([4, 2])) == EX["fig6_after_O2_digits"][1]
    lay = _eq2()
    assert lay.apply([4, 2]) == EX["fig6_apply"][1]
    assert L.canon_unflatten([2, 2, 3, 3], lay.apply([4, 2])) == EX["fig6_apply_digits"][1]
    assert lay.inv(15) == EX["fig6_inv"][1]


def test_chain_order_reversed_differs():
    """The opposite reading of chain order gives a different value (17), so the
    Figure 6 pin really decides the order."""
    o2 = L.OrderBy(L.RegP([2, 3, 2, 3], [1, 3, 2, 4]))
    o1 = L.OrderBy(L.RegP([2, 2], [2, 1]), L.antidiag_genp(3))
    rev = L.GroupBy([6, 6], chain=[o1, o2])
    assert rev.apply([4, 2]) == 17


def test_sigma_dq_printed():
    assert L.sigma_dq(2, 3) == EX["sigma_2x3"][1]
    assert L.sigma_dq(3, 2) == EX["sigma_3x2"][1]
    assert L.sigma_inverse(L.sigma_dq(2, 3)) == L.sigma_dq(3, 2)


def test_tileby_physical_spaces_printed():
    """Applying sigma_{2x3} / sigma_{3x2} to the logical dims gives the
    physical spaces printed after the sugar definitions."""
    n = ["n11", "n12", "n21", "n22", "n31", "n32"]  # TileBy_{3x2}: 3 levels of 2 dims
    assert L.sigma_gather(L.sigma_dq(2, 3), n) == ["n11", "n21", "n31", "n12", "n22", "n32"]
    n = ["n11", "n12", "n13", "n21", "n22", "n23"]  # TileBy_{2x3}
    assert L.sigma_gather(L.sigma_dq(3, 2), n) == ["n11", "n21", "n12", "n22", "n13", "n23"]


# ---------------------------------------------------------------- antidiag
def test_antidiag_n3_table():
    tab = [[L.antidiag(3, i, j) for j in range(3)] for i in range(3)]
    assert tab == [[0, 1, 3], [2, 4, 6], [5, 7, 8]]


@pytest.mark.parametrize("n", list(range(1, 65)))
def test_antidiag_bijection_and_inverse(n):
    i, j = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    z = L.antidiag(n, i.ravel(), j.ravel())
    assert sorted(z.tolist()) == list(range(n * n))
    ii, jj = L.antidiag_inv(n, z)
    assert (ii == i.ravel()).all() and (jj == j.ravel()).all()
    # antidiagonals are filled in order: a smaller i+j never comes later
    order = np.argsort(z)
    s = (i.ravel() + j.ravel())[order]
    assert (np.diff(s) >= 0).all()


@pytest.mark.parametrize("n", [1, 2, 3, 5, 8, 12])
def test_antidiag_equals_brute_force_ranking(n):
    """Figure 7's order by brute force: rank every (i, j) of the tile by
    (antidiagonal i + j, then row i); the rank is the number."""
    pts = sorted(((i + j, i), (i, j)) for i in range(n) for j in range(n))
    for rank, (_, (i, j)) in enumerate(pts):
        assert int(L.antidiag(n, i, j)) == rank
        assert [int(v) for v in L.antidiag_inv(n, rank)] == [i, j]


def test_antidiag_figure6_value():
    """Figure 6's walk-through lands on 15 = block 1, element 6: element (1, 2)
    of a 3 x 3 block in antidiagonal order is 6."""
    assert int(L.antidiag(3, 1, 2)) == 6


# ------------------------------------------------------------ Table I rows
@pytest.mark.parametrize("M,K,BM,BK", [(8, 12, 4, 3), (16, 8, 4, 4), (6, 10, 3, 5)])
def test_table1_tileby_row_is_cute_strides(M, K, BM, BK):
    lay = L.TileBy([M // BM, K // BK], [BM, BK]).OrderBy(L.Row(M, K))
    for tm, tk, im, ik in itertools.product(range(M // BM), range(K // BK), range(BM), range(BK)):
        assert lay.apply([tm, tk, im, ik]) == tm * K * BM + tk * BK + im * K + ik


def test_table1_fig6_mid_inverse_strides():
    lay = L.GroupBy([6, 6]).OrderBy(L.RegP([2, 3, 2, 3], [1, 3, 2, 4]))
    for bi, bj, ii, jj in itertools.product(range(2), range(2), range(3), range(3)):
        phys = L.canon_flatten([2, 2, 3, 3], [bi, bj, ii, jj])
        assert L.canon_flatten([6, 6], lay.inv(phys)) == 18 * bi + 3 * bj + 6 * ii + jj


@pytest.mark.parametrize("R_,T", [(2, 3), (4, 4), (3, 2)])
def test_table1_lud_row(R_, T):
    lay = L.GroupBy([R_, R_], [T, T]).OrderBy(L.Row(R_ * T, R_ * T))
    for a, b, c, d in itertools.product(range(R_), range(R_), range(T), range(T)):
        assert lay.apply([a, b, c, d]) == a * R_ * T * T + b * T * T + c * T + d


def test_fig8_colour_classes():
    lay = L.GroupBy([2, 2, 2, 2, 2]).OrderBy(L.RegP([2] * 5, [5, 2, 4, 3, 1]))
    classes = {}
    with open(os.path.join(GOLDEN, "fig8_layout.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            row, col, label, colour = line.split()
            row, col, label = int(row), int(col), int(label)
            assert label == 4 * col + row
            classes.setdefault(colour, []).append(label)
    blocks = {}
    for colour, labels in classes.items():
        phys = sorted(lay.apply(L.canon_unflatten([2] * 5, x)) for x in labels)
        assert phys == list(range(phys[0], phys[0] + 8)) and phys[0] % 8 == 0
        blocks[colour] = phys[0] // 8
    assert sorted(blocks.values()) == [0, 1, 2, 3]


# -------------------------------------------------------------------- Col
@pytest.mark.parametrize("M,K,BM,BK", [(8, 12, 4, 3), (6, 4, 2, 2)])
def test_col_reading_is_column_major(M, K, BM, BK):
    lay = L.TileBy([M // BM, K // BK], [BM, BK]).OrderBy(L.Col(M, K))
    for tm, tk, im, ik in itertools.product(range(M // BM), range(K // BK), range(BM), range(BK)):
        m, k = tm * BM + im, tk * BK + ik
        assert lay.apply([tm, tk, im, ik]) == k * M + m


def test_col_literal_formula_is_not_column_major():
    """The printed Col (dims reversed too) fails column-major on M != K, which
    is why the reading keeps the logical dims."""
    M, K = 6, 4
    literal = L.RegP([K, M], [2, 1])  # RegP([n_d..n_1],[d..1])
    ok = all(L.as_layout(literal).apply([m, k]) == k * M + m
             for m in range(K) for k in range(M))
    assert not ok


# ------------------------------------------------------------ TileOrderBy
def test_tileorderby_c1_closed_form():
    lay = L.TileOrderBy(L.Row(2, 2), L.Row(4, 4), L.Row(16, 16))
    r, c = np.meshgrid(np.arange(128), np.arange(128), indexing="ij")
    r, c = r.ravel(), c.ravel()
    exp = ((((r >> 6) * 2 + (c >> 6)) * 4 + ((r >> 4) & 3)) * 4 + ((c >> 4) & 3)) * 256 \
        + (r & 15) * 16 + (c & 15)
    assert (lay.apply([r, c]) == exp).all()


def test_tileorderby_c2_closed_form_sampled():
    lay = L.TileOrderBy(L.Col(128, 128), L.Row(64, 64))
    rng = np.random.default_rng(0)
    r = rng.integers(0, 8192, 200000)
    c = rng.integers(0, 8192, 200000)
    exp = ((c // 64) * 128 + r // 64) * 4096 + (r % 64) * 64 + c % 64
    assert (lay.apply([r, c]) == exp).all()


def test_tileby_tileorderby_are_mutual_inverses():
    """TileBy maps tile coordinates to the row-major position; TileOrderBy of
    Rows maps full coordinates to tile-major storage.  Composing one with the
    other is the identity on tile-major digits."""
    tb = L.TileBy([2, 3], [4, 2])          # logical [2,3,4,2] -> row-major of [8,6]
    to = L.TileOrderBy(L.Row(2, 3), L.Row(4, 2))
    for x in range(48):
        digits = L.canon_unflatten([2, 3, 4, 2], x)
        rm = tb.apply(digits)
        r, c = divmod(rm, 6)
        assert to.apply([r, c]) == x


# ------------------------------------------------------------------ Morton
def test_morton_2x2_is_z():
    lay = L.as_layout(L.morton_genp(2, 2))
    assert [[lay.apply([i, j]) for j in range(2)] for i in range(2)] == [[0, 1], [2, 3]]


def test_morton_4x4_brute_force():
    # Z-order of a 4x4 grid, written out from the bit-interleaving definition.
    exp = [[0, 1, 4, 5], [2, 3, 6, 7], [8, 9, 12, 13], [10, 11, 14, 15]]
    lay = L.as_layout(L.morton_genp(4, 4))
    assert [[lay.apply([i, j]) for j in range(4)] for i in range(4)] == exp


@pytest.mark.parametrize("s", [1, 2, 3, 4, 5, 6])
def test_morton_equals_recursive_2x2_tiling(s):
    """Z-order is recursive 2x2 tiling: GenP(morton) over 2^s x 2^s equals
    TileOrderBy of s levels of Row[2,2] (a second, independent formulation)."""
    n = 1 << s
    z = L.as_layout(L.morton_genp(n, n))
    t = L.TileOrderBy(*[L.Row(2, 2) for _ in range(s)])
    r, c = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    assert (np.asarray(z.apply([r.ravel(), c.ravel()])) == t.apply([r.ravel(), c.ravel()])).all()


def test_morton_aligned_squares_contiguous_and_rows_runs_of_two():
    n = 64
    lay = L.as_layout(L.morton_genp(n, n))
    for s in (1, 2, 3, 4):
        w = 1 << s
        for bi in range(0, n, w * 3):
            for bj in range(0, n, w * 5):
                v = sorted(lay.apply([i, j]) for i in range(bi, bi + w) for j in range(bj, bj + w))
                assert v == list(range(v[0], v[0] + w * w)) and v[0] % (w * w) == 0
    row = [lay.apply([5, j]) for j in range(n)]
    runs = [row[k + 1] - row[k] == 1 for k in range(n - 1)]
    assert runs[0::2] == [True] * (n // 2) and not any(runs[1::2])


def test_morton_nonsquare_bijection():
    lay = L.as_layout(L.morton_genp(4, 16))
    vals = sorted(lay.apply([i, j]) for i in range(4) for j in range(16))
    assert vals == list(range(64))
    for x in range(64):
        assert lay.apply(lay.inv(x)) == x


# ------------------------------------------------------------- XOR swizzle
@pytest.mark.parametrize("R_,C,v,s", [(256, 64, 8, 1), (128, 32, 8, 2), (64, 64, 4, 1), (16, 16, 2, 4)])
def test_xor_swizzle_bijection(R_, C, v, s):
    g = L.xor_swizzle_genp(R_, C, v, s)
    lay = L.as_layout(g)
    x = L.apply_all(lay)
    assert (np.sort(x) == np.arange(R_ * C)).all()
    inv = L.inv_all(lay)
    r, c = np.divmod(np.arange(R_ * C), C)
    assert (inv[x, 0] == r).all() and (inv[x, 1] == c).all()
    # rows stay rows, vectors of v stay contiguous and aligned
    assert (x // C == r).all()
    assert ((x % v) == (c % v)).all()


def test_xor_swizzle_reduces_to_row():
    R_, C = 8, 32
    g = L.as_layout(L.xor_swizzle_genp(R_, C, 8, 64))  # s > R: r/s = 0
    r, c = np.divmod(np.arange(R_ * C), C)
    assert (L.apply_all(g) == r * C + c).all()


def test_xor_swizzle_spreads_a_column_over_banks():
    """Vector v of column group 0 moves to a different slot in each of C/v rows."""
    R_, C, v = 64, 64, 8
    g = L.as_layout(L.xor_swizzle_genp(R_, C, v, 1))
    slots = [(g.apply([r, 0]) % C) // v for r in range(C // v)]
    assert sorted(slots) == list(range(C // v))


# ------------------------------------------------- grouped tile schedule
def _group_rule(pid, mt, nt, g):
    """Grouped program-id order (Section II): groups of g tile-rows, column-
    major inside a group, groups in order."""
    group = pid // (g * nt)
    first = group * g
    size = min(mt - first, g)
    return first + (pid % (g * nt)) % size, (pid % (g * nt)) // size


@pytest.mark.parametrize("mt,nt,g", [(8, 8, 8), (32, 32, 8), (16, 4, 4), (6, 5, 3)])
def test_grouped_schedule_layout(mt, nt, g):
    sched = L.GroupBy([mt, nt]).OrderBy(L.RegP([mt // g, g, nt], [1, 3, 2]))
    for pid in range(mt * nt):
        assert tuple(sched.inv(pid)) == _group_rule(pid, mt, nt, g)


def test_xcd_remap_composition_bijective():
    p = 1024
    xcd = L.GroupBy([p // 8, 8]).OrderBy(L.RegP([p // 8, 8], [2, 1]))
    sched = L.GroupBy([32, 32]).OrderBy(L.RegP([4, 8, 32], [1, 3, 2]))
    seen = set()
    for b in range(p):
        q = xcd.apply(L.canon_unflatten([p // 8, 8], b))
        assert q == (b % 8) * (p // 8) + b // 8
        seen.add(tuple(sched.inv(q)))
    assert len(seen) == p


# --------------------------------------------------- bijection invariants
def _random_layout(rng):
    """A random GroupBy chain over a tiny space, built from RegP / GenP pieces."""
    shape = [int(x) for x in rng.choice([2, 3, 4], size=2)]
    n = shape[0] * shape[1]
    chain = []
    for _ in range(rng.integers(1, 4)):
        # factor n into 1-3 pieces of 1-3 dims each
        pieces = []
        rem = n
        while rem > 1:
            f = [x for x in (2, 3, 4, 6, 8, 9) if rem % x == 0]
            a = int(rng.choice(f))
            b = [x for x in (1, 2, 3) if a % x == 0]
            d0 = int(rng.choice(b))
            dims = [d0, a // d0]
            kind = rng.integers(0, 3)
            if kind == 0:
                pieces.append(L.RegP(dims, list(rng.permutation([1, 2]) )))
            elif kind == 1:
                pieces.append(L.reverse_genp(*dims))
            else:
                pieces.append(L.Row(dims))
            rem //= a
        if not pieces:
            pieces = [L.Row(1, 1)]
        chain.append(L.OrderBy(*pieces))
    return L.GroupBy(shape, chain=chain)


def test_random_layouts_are_bijections():
    rng = np.random.default_rng(1)
    for _ in range(200):
        lay = _random_layout(rng)
        n = lay.size()
        phys = [lay.apply(L.canon_unflatten(lay.dims(), x)) for x in range(n)]
        assert sorted(phys) == list(range(n))
        for x in range(n):
            assert L.canon_flatten(lay.dims(), lay.inv(phys[x])) == x


def test_expandby_partial_tiles():
    """ExpandBy (Figure 9): a 5x7 array tiled by 2x4 tiles inside 6x8."""
    g = L.TileOrderBy(L.Row(3, 2), L.Row(2, 4))  # over [6, 8]
    e = L.ExpandBy([5, 7], [6, 8], g)
    seen = []
    for i in range(6):
        for j in range(8):
            v = e.apply([i, j])
            # g sends (i,j) to tile-major storage; decode back to check the rule
            ip = L.canon_unflatten([6, 8], g.apply([i, j]))
            exp = ip[0] * 7 + ip[1] if (ip[0] < 5 and ip[1] < 7) else -1
            assert v == exp
            if v >= 0:
                seen.append(v)
                assert L.canon_flatten([6, 8], e.inv(v)) == L.canon_flatten([6, 8], [i, j])
    assert sorted(seen) == list(range(35))


# ------------------------------------------------------------------- remap
def test_remap_transpose_matches_numpy():
    n, m = 12, 20
    src = np.arange(n * m, dtype=np.float32)
    out = R.remap(L.as_layout(L.Row(n, m)), L.as_layout(L.Col(n, m)), src)
    assert (out == src.reshape(n, m).T.ravel()).all()


def test_remap_expandby_pads_and_crops_like_numpy():
    """ExpandBy source (Figure 9): the compact 5x7 array lands in a 6x8 tiled
    buffer with zero padding, equal to numpy's pad followed by the tile-major
    reshape; the ExpandBy destination crops it back."""
    data = np.arange(1, 36, dtype=np.int32)
    src = L.ExpandBy([5, 7], [6, 8], L.as_layout(L.Row(6, 8)))
    tiled = L.TileOrderBy(L.Row(3, 2), L.Row(2, 4))  # 2x4 tiles over [6, 8]
    out = R.remap(src, tiled, data)
    padded = np.pad(data.reshape(5, 7), ((0, 1), (0, 1)))
    assert (out == padded.reshape(3, 2, 2, 4).transpose(0, 2, 1, 3).ravel()).all()
    back = R.remap(tiled, src, out)
    assert (back == data).all()
    # row-major padding alone is numpy's pad, and a fill value is honoured
    out2 = R.remap(src, L.as_layout(L.Row(6, 8)), data, fill=-7)
    assert (out2 == np.pad(data.reshape(5, 7), ((0, 1), (0, 1)), constant_values=-7).ravel()).all()


def test_remap_blocked_matches_numpy_reshape():
    """Row -> 2-level blocked (column-major tile order, row-major tiles) equals
    a numpy reshape/transpose of the same data."""
    n, t = 32, 8
    src = np.arange(n * n, dtype=np.int32)
    lay = L.TileOrderBy(L.Col(n // t, n // t), L.Row(t, t))
    out = R.remap(L.as_layout(L.Row(n, n)), lay, src)
    blocks = src.reshape(n // t, t, n // t, t).transpose(2, 0, 1, 3)  # [cb, rb, r, c]
    assert (out == blocks.ravel()).all()


def test_remap_3d_bricks_match_numpy_reshape():
    """TileOrderBy of two 3-D Row pieces stores a grid as bricks (the 3-D
    subdomains of Section V's stencil layout), bricks in row-major order,
    row-major inside each brick: a 6-D reshape/transpose of the row-major
    array.  With ExpandBy, a grid the bricks do not divide is zero-padded."""
    nb, b = (3, 2, 4), (2, 5, 3)
    n = [x * y for x, y in zip(nb, b)]
    src = np.arange(int(np.prod(n)), dtype=np.int64)
    bricks = L.TileOrderBy(L.Row(*nb), L.Row(*b))
    out = R.remap(L.as_layout(L.Row(*n)), bricks, src)
    exp = src.reshape(nb[0], b[0], nb[1], b[1], nb[2], b[2]).transpose(0, 2, 4, 1, 3, 5)
    assert (out == exp.ravel()).all()
    assert (R.remap(bricks, L.as_layout(L.Row(*n)), out) == src).all()
    m = [5, 9, 10]  # padded to n = [6, 10, 12]
    data = np.arange(1, int(np.prod(m)) + 1, dtype=np.int64)
    out = R.remap(L.ExpandBy(m, n, L.as_layout(L.Row(*n))), bricks, data)
    padded = np.pad(data.reshape(m), [(0, x - y) for x, y in zip(n, m)])
    exp = padded.reshape(nb[0], b[0], nb[1], b[1], nb[2], b[2]).transpose(0, 2, 4, 1, 3, 5)
    assert (out == exp.ravel()).all()


def test_remap_inverse_roundtrip_and_multiset():
    rng = np.random.default_rng(2)
    a = L.as_layout(L.Row(16, 16))
    b = L.as_layout(L.morton_genp(16, 16))
    src = rng.standard_normal(256).astype(np.float32)
    fwd = R.remap(a, b, src)
    back = R.remap(b, a, fwd)
    assert (back == src).all()
    assert sorted(fwd.tolist()) == sorted(src.tolist())


# -------------------------------------------------------------------- gemm
def _f16(x):
    return np.asarray(x, dtype=np.float16).view(np.uint16)


def _bf16(x):
    b = np.asarray(x, dtype=np.float32).view(np.uint32)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)


def test_gemm_small_integers_exact():
    rng = np.random.default_rng(3)
    m, n, k = 16, 24, 40
    a = rng.integers(-2, 3, (m, k))
    b = rng.integers(-2, 3, (k, n))
    la, lb = L.as_layout(L.Row(m, k)), L.as_layout(L.Col(k, n))
    abuf = _f16(a.ravel())
    bbuf = _f16(b.T.ravel())  # column-major storage of B
    r = G.gemm(abuf, bbuf, la, lb, "f16")
    assert (r == (a @ b)).all()


def test_gemm_bf16_decode_and_layouts():
    rng = np.random.default_rng(4)
    m, n, k = 8, 12, 16
    a = rng.standard_normal((m, k)).astype(np.float32)
    b = rng.standard_normal((k, n)).astype(np.float32)
    abits, bbits = _bf16(a.ravel()), _bf16(b.ravel())
    ad = (abits.astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(m, k)
    bd = (bbits.astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(k, n)
    r = G.gemm(abits, bbits, L.as_layout(L.Row(m, k)), L.as_layout(L.Row(k, n)), "bf16")
    assert np.allclose(r, ad @ bd, rtol=0, atol=1e-12)
    assert np.abs(ad - a).max() <= np.abs(a).max() * 2 ** -8


def test_gemm_morton_operand():
    n = 16
    rng = np.random.default_rng(5)
    a = rng.integers(-2, 3, (n, n))
    b = rng.integers(-2, 3, (n, n))
    mz = L.as_layout(L.morton_genp(n, n))
    abuf = np.empty(n * n, dtype=np.float16)
    for i in range(n):
        for j in range(n):
            abuf[mz.apply([i, j])] = a[i, j]
    r = G.gemm(abuf.view(np.uint16), _f16(b.ravel()), mz, L.as_layout(L.Row(n, n)), "f16")
    assert (r == a @ b).all()


def test_tolerance_helper():
    r = np.array([[1.0, -2.0], [1e-6, 4.0]])
    ok, mre, fre = G.check_tolerance(r * (1 + 1e-4), r)
    assert ok and mre < 2e-4
    ok, _, _ = G.check_tolerance(r + np.array([[0, 0], [0.5, 0]]), r)
    assert not ok


# --------------------------------------------------------- planted mistakes
def _expect_pins_fail(monkeypatch, target, name, bad):
    monkeypatch.setattr(target, name, bad)
    failures = 0
    for t in (test_fig2_worked_example, test_fig6_eq2_worked_example, test_tileorderby_c1_closed_form,
              lambda: test_table1_tileby_row_is_cute_strides(8, 12, 4, 3),
              lambda: test_grouped_schedule_layout(8, 8, 4)):
        try:
            t()
        except (AssertionError, Exception):
            failures += 1
    return failures


def test_planted_unflatten_first_fastest_is_caught(monkeypatch):
    def bad(n, x):
        out = []
        for nk in n:
            out.append(x % int(nk))
            x = x // int(nk)
        return out
    assert _expect_pins_fail(monkeypatch, L, "canon_unflatten", bad) > 0


def test_planted_sigma_scatter_is_caught(monkeypatch):
    def bad(sigma, v):  # scatter instead of gather
        out = [None] * len(sigma)
        for k, s in enumerate(sigma):
            out[s - 1] = v[k]
        return out
    assert _expect_pins_fail(monkeypatch, L, "sigma_gather", bad) > 0


def test_planted_orderby_wrong_accumulate_is_caught(monkeypatch):
    def bad_apply(self, idx):
        flat, pos = 0, 0
        for p in self.pieces:
            d = len(p.dims())
            flat = flat + p.apply(idx[pos:pos + d]) * p.size()  # wrong Horner step
            pos += d
        return flat
    assert _expect_pins_fail(monkeypatch, L.OrderBy, "apply", bad_apply) > 0


def test_planted_chain_order_is_caught(monkeypatch):
    def bad_apply(self, idx):
        flat = L.canon_flatten(self.dims(), list(idx))
        for o in reversed(self.chain):
            flat = o.apply(L.canon_unflatten(o.dims(), flat))
        return flat
    assert _expect_pins_fail(monkeypatch, L.GroupBy, "apply", bad_apply) > 0


def test_planted_antidiag_sign_is_caught():
    def bad(n, i, j):
        a = i + j + 1
        return i + (a * (a - 1)) // 2 if a <= n else n * n - n + j - ((2 * n - a) * (2 * n - a - 1)) // 2
    tab = [[bad(3, i, j) for j in range(3)] for i in range(3)]
    assert tab != [[0, 1, 3], [2, 4, 6], [5, 7, 8]]


def test_planted_transposed_gemm_operand_is_caught():
    rng = np.random.default_rng(6)
    m = 6
    a = rng.integers(-2, 3, (m, m))
    b = rng.integers(-2, 3, (m, m))
    # B stored row-major but described as Col: the product must differ
    r = G.gemm(_f16(a.ravel()), _f16(b.ravel()), L.as_layout(L.Row(m, m)), L.as_layout(L.Col(m, m)), "f16")
    assert not (r == a @ b).all()


# ------------------------------------------------- expression GenP (oracle)
from oracle import genexpr as GX  # noqa: E402
from tests import genp_exprs as GE  # noqa: E402


@pytest.mark.parametrize("text,value", [
    ("1 + 2 * 3 << 1", 14), ("5 - 3 - 1", 1), ("2 ^ 3 & 1", 3), ("0 - 7 / 2", -3), ("-7 / 2", -4),
    ("-7 % 2", 1), ("1 < 2 == 1", 1), ("0 ? 5 : 1 ? 6 : 7", 6), ("isqrt(99)", 9), ("isqrt(100)", 10),
    ("max(3, min(9, 4))", 4), ("!0 + !5", 1), ("1 && 0 || 1", 1), ("3 >= 3 && 2 > 3", 0), ("6 != 6", 0),
])
def test_expression_language_follows_c_rules(text, value):
    """Precedence, associativity and floor division of the expression
    language, on values worked out by hand from C's rules."""
    assert int(GX.evaluate(text)) == value


def test_expression_antidiag_equals_figure7():
    """The antidiagonal order written as an expression equals the Figure 7
    permutation (pinned above) for n = 1..12, forward and inverse."""
    for n in range(1, 13):
        g = GX.expr_genp([n, n], GE.ANTIDIAG_APPLY, GE.ANTIDIAG_INV)
        ref = L.antidiag_genp(n)
        i, j = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
        assert (g.apply([i, j]) == ref.apply([i, j])).all()
        x = np.arange(n * n)
        assert all((a == b).all() for a, b in zip(g.inv(x), ref.inv(x)))


def test_expression_morton_and_row_col():
    """Bit-level Z order equals GenP(morton) on 8x8; i*n1+j and j*n0+i equal
    Row and Col."""
    i, j = np.meshgrid(np.arange(8), np.arange(8), indexing="ij")
    g = GX.expr_genp([8, 8], GE.MORTON8_APPLY, GE.MORTON8_INV)
    assert (g.apply([i, j]) == L.morton_genp(8, 8).apply([i, j])).all()
    x = np.arange(64)
    assert all((a == b).all() for a, b in zip(g.inv(x), L.morton_genp(8, 8).inv(x)))
    i, j = np.meshgrid(np.arange(5), np.arange(7), indexing="ij")
    row = GX.expr_genp([5, 7], "i * n1 + j", ["x / n1", "x % n1"])
    col = GX.expr_genp([5, 7], "i1 * n0 + i0", ["x % n0", "x / n0"])
    assert (row.apply([i, j]) == L.Row(5, 7).apply([i, j])).all()
    assert (col.apply([i, j]) == L.Col(5, 7).apply([i, j])).all()
    s = GX.expr_genp([256, 64], GE.SWIZZLE64_APPLY, GE.SWIZZLE64_INV)
    i, j = np.meshgrid(np.arange(256), np.arange(64), indexing="ij")
    assert (s.apply([i, j]) == L.xor_swizzle_genp(256, 64, 8, 2).apply([i, j])).all()


def test_byte_pattern_slices_agree():
    """The large-buffer byte generator: any slice equals the values at those
    indices, beyond 2^32 too, and the bytes are spread over 0..255."""
    import synth_inputs as S
    for start in (0, (1 << 32) - 100, 5 << 32):
        a = S.byte_pattern(start, 1000).numpy()
        assert (a == S.byte_pattern_at(np.arange(start, start + 1000))).all()
    v = S.byte_pattern(0, 1 << 16).numpy()
    assert len(np.unique(v)) == 256 and abs(v.mean() - 127.5) < 3
