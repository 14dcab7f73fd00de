"""Remaps on the GPU must equal the oracle byte for byte."""
import numpy as np
import pytest

import synth_inputs as S
from oracle import layout as OL
from oracle import remap as OR
from tests.gpu_util import bits, need_gpu, say

pytestmark = pytest.mark.gpu


def _run(lego, src_l, dst_l, src, dev):
    import torch
    d_src = src.to(dev)
    d_dst = torch.empty_like(d_src)
    lego.remap(src_l, dst_l, d_src, d_dst)
    torch.cuda.synchronize()
    return d_dst.cpu()


def test_remap_c2_row_blocked_roundtrip(lego):
    """8192^2 fp32 Row -> blocked (64x64 tiles, column-major tile order) and back."""
    dev = need_gpu()
    n = 8192
    src = S.tensor(n * n, "f32", seed=S.SEED_SRC)
    row, blk = lego.as_layout(lego.Row(n, n)), lego.TileOrderBy(lego.Col(128, 128), lego.Row(64, 64))
    orow, oblk = OL.as_layout(OL.Row(n, n)), OL.TileOrderBy(OL.Col(128, 128), OL.Row(64, 64))
    say(f"remap C2 fwd plan={lego.remap_plan(row, blk, 4)['info']}")
    fwd = _run(lego, row, blk, src, dev)
    exp = OR.remap(orow, oblk, src.numpy())
    assert (bits(fwd) == exp.view(np.uint32)).all()
    say(f"remap C2 inv plan={lego.remap_plan(blk, row, 4)['info']}")
    back = _run(lego, blk, row, fwd, dev)
    assert (bits(back) == bits(src)).all()


def test_remap_c5_row_morton_roundtrip(lego):
    """4096^2 fp16 Row -> Morton and back (LDS-staged path)."""
    dev = need_gpu()
    n = 4096
    src = S.tensor(n * n, "f16", seed=S.SEED_SRC)
    row, mz = lego.as_layout(lego.Row(n, n)), lego.as_layout(lego.GenP("morton", [n, n]))
    orow, omz = OL.as_layout(OL.Row(n, n)), OL.as_layout(OL.morton_genp(n, n))
    say(f"remap C5 row->morton plan={lego.remap_plan(row, mz, 2)['info']}")
    fwd = _run(lego, row, mz, src, dev)
    exp = OR.remap(orow, omz, S.as_numpy_bits(src))
    assert (bits(fwd) == exp).all()
    say(f"remap C5 morton->row plan={lego.remap_plan(mz, row, 2)['info']}")
    back = _run(lego, mz, row, fwd, dev)
    assert (bits(back) == bits(src)).all()


@pytest.mark.parametrize("n,dtype", [(2048, "f32"), (4096, "f32"), (8192, "f32"), (4096, "f16"), (1024, "bf16")])
def test_remap_transpose(lego, n, dtype):
    """Row -> Col and Col -> Row (the transpose of Table V), each direction on
    its own source, every element against the oracle's remap.  The fp32
    sizes are the measured ones; 4096^2 and 8192^2 take the 64 KiB tiles read
    in source order, which the plan text must show."""
    dev = need_gpu()
    row, col = lego.as_layout(lego.Row(n, n)), lego.as_layout(lego.Col(n, n))
    orow, ocol = OL.as_layout(OL.Row(n, n)), OL.as_layout(OL.Col(n, n))
    for seed, (ls, ld, ols, old, name) in enumerate(((row, col, orow, ocol, "row->col"),
                                                     (col, row, ocol, orow, "col->row"))):
        src = S.tensor(n * n, dtype, seed=S.SEED_SRC + seed)
        info = lego.remap_plan(ls, ld, src.element_size())["info"]
        say(f"remap transpose {name} n={n} {dtype} plan={info}")
        if dtype == "f32" and n >= 4096:
            assert info.startswith("lds TILE=16384 ") and " src-order " in info, info
        out = _run(lego, ls, ld, src, dev)
        exp = OR.remap(ols, old, bits(src))
        assert (bits(out) == exp).all(), name


@pytest.mark.parametrize("n,dtype", [(4096, "f32"), (8192, "f32"), (4096, "f16")])
def test_remap_antidiagonal_full(lego, n, dtype):
    """Row -> antidiagonal order (Figure 7's GenP over the whole matrix) and
    back, each direction on its own source, every element against the
    oracle's remap: the box plans the bench measures (128 x 128 boxes beyond
    the last-level cache, the forward walking its rectangle of boxes in
    bands)."""
    dev = need_gpu()
    row, ad = lego.as_layout(lego.Row(n, n)), lego.as_layout(lego.GenP("antidiag", [n, n]))
    orow, oad = OL.as_layout(OL.Row(n, n)), OL.as_layout(OL.antidiag_genp(n))
    for seed, (ls, ld, ols, old, name) in enumerate(((row, ad, orow, oad, "row->antidiag"),
                                                     (ad, row, oad, orow, "antidiag->row"))):
        src = S.tensor(n * n, dtype, seed=S.SEED_SRC + seed)
        info = lego.remap_plan(ls, ld, src.element_size())["info"]
        say(f"remap antidiagonal {name} n={n} {dtype} plan={info}")
        assert info.startswith("box "), info
        if n == 8192 and seed == 0:
            assert info.startswith("box 128x128 tiles32-bands4-xcd "), info
        out = _run(lego, ls, ld, src, dev)
        exp = OR.remap(ols, old, bits(src))
        assert (bits(out) == exp).all(), name


@pytest.mark.parametrize("b", [8, 4])
def test_remap_bricks_512cubed_sampled(lego, b):
    """512^3 fp32 Row <-> bricks of b^3 (the configuration the bench times):
    200k sampled destination elements against the oracle's inverse, then the
    round trip back to row-major must be the identity."""
    import torch
    dev = need_gpu()
    n = 512
    src = S.tensor(n ** 3, "f32", seed=S.SEED_SRC)
    row, br = lego.as_layout(lego.Row(n, n, n)), lego.TileOrderBy(lego.Row(n // b, n // b, n // b), lego.Row(b, b, b))
    obr, orow = OL.TileOrderBy(OL.Row(n // b, n // b, n // b), OL.Row(b, b, b)), OL.as_layout(OL.Row(n, n, n))
    say(f"remap bricks {b}^3 of 512^3 plan={lego.remap_plan(row, br, 4)['info']}")
    out = _run(lego, row, br, src, dev)
    p = np.random.default_rng(b).integers(0, n ** 3, 200000)
    q = orow.apply(obr.inv(p))
    sb = bits(src)
    assert (bits(out)[p] == sb[q]).all()
    say(f"remap bricks {b}^3 of 512^3 back plan={lego.remap_plan(br, row, 4)['info']}")
    back = _run(lego, br, row, out, dev)
    assert (bits(back) == sb).all()


def test_remap_beyond_4g_elements(lego):
    """65600^2 one-byte elements (more than 2^32; 65600 = 64 * 1025): Row to
    64x64 blocked (direct path) and Row to Col (LDS path, 64-bit offsets).
    The first and last 4096 and 10^6 random destination elements against the
    oracle, then the round trip back must be the identity."""
    import torch
    dev = need_gpu()
    n = 65600
    N = n * n
    src = torch.empty(N, dtype=torch.uint8, device=dev)
    for s0 in range(0, N, 1 << 28):
        c = min(1 << 28, N - s0)
        src[s0:s0 + c] = S.byte_pattern(s0, c, device=dev)
    rng = np.random.default_rng(5)
    p = np.concatenate([np.arange(4096), N - 4096 + np.arange(4096), rng.integers(0, N, 1_000_000)])
    pt = torch.from_numpy(p).to(dev)
    row, orow = lego.as_layout(lego.Row(n, n)), OL.as_layout(OL.Row(n, n))
    for name, ld, old in (
            ("blocked", lego.TileOrderBy(lego.Col(n // 64, n // 64), lego.Row(64, 64)),
             OL.TileOrderBy(OL.Col(n // 64, n // 64), OL.Row(64, 64))),
            ("col", lego.as_layout(lego.Col(n, n)), OL.as_layout(OL.Col(n, n)))):
        say(f"remap 65600^2 u8 row->{name} plan={lego.remap_plan(row, ld, 1)['info']}")
        dst = torch.empty_like(src)
        lego.remap(row, ld, src, dst)
        torch.cuda.synchronize()
        exp = S.byte_pattern_at(orow.apply(old.inv(p)))
        assert (dst[pt].cpu().numpy() == exp).all(), name
        say(f"remap 65600^2 u8 {name}->row plan={lego.remap_plan(ld, row, 1)['info']}")
        back = torch.empty_like(src)
        lego.remap(ld, row, dst, back)
        torch.cuda.synchronize()
        assert torch.equal(back, src), name
        del dst, back


def _small_cases(L):
    return [
        ("antidiag chain 6x6 (gather)",
         L.as_layout(L.Row(6, 6)),
         L.GroupBy([6, 6]).OrderBy(L.RegP([2, 3, 2, 3], [1, 3, 2, 4])).OrderBy(L.RegP([2, 2], [2, 1]),
                                                                             L.GenP("antidiag", [3, 3])),
         OL.as_layout(OL.Row(6, 6)),
         OL.GroupBy([6, 6]).OrderBy(OL.RegP([2, 3, 2, 3], [1, 3, 2, 4])).OrderBy(OL.RegP([2, 2], [2, 1]),
                                                                               OL.antidiag_genp(3))),
        ("ragged 3x5 tiles of 7x3", L.as_layout(L.Row(21, 15)), L.TileOrderBy(L.Col(3, 5), L.Row(7, 3)),
         OL.as_layout(OL.Row(21, 15)), OL.TileOrderBy(OL.Col(3, 5), OL.Row(7, 3))),
        ("xor swizzle 256x64", L.as_layout(L.Row(256, 64)), L.as_layout(L.GenP("xor_swizzle", [256, 64], [8, 1])),
         OL.as_layout(OL.Row(256, 64)), OL.as_layout(OL.xor_swizzle_genp(256, 64, 8, 1))),
        ("morton 16x16 vs col", L.as_layout(L.Col(16, 16)), L.as_layout(L.GenP("morton", [16, 16])),
         OL.as_layout(OL.Col(16, 16)), OL.as_layout(OL.morton_genp(16, 16))),
        ("identity 1x1", L.as_layout(L.Row(1, 1)), L.as_layout(L.Row(1, 1)),
         OL.as_layout(OL.Row(1, 1)), OL.as_layout(OL.Row(1, 1))),
        ("odd 1000x3 to col", L.as_layout(L.Row(1000, 3)), L.as_layout(L.Col(1000, 3)),
         OL.as_layout(OL.Row(1000, 3)), OL.as_layout(OL.Col(1000, 3))),
        ("3-level blocked 512^2", L.as_layout(L.Row(512, 512)),
         L.TileOrderBy(L.Col(4, 4), L.Row(4, 4), L.Row(32, 32)),
         OL.as_layout(OL.Row(512, 512)), OL.TileOrderBy(OL.Col(4, 4), OL.Row(4, 4), OL.Row(32, 32))),
        # transposes whose extents are not powers of two (LDS tiles of odd sizes,
        # workgroups that are not whole waves)
        ("transpose 1000x1000", L.as_layout(L.Row(1000, 1000)), L.as_layout(L.Col(1000, 1000)),
         OL.as_layout(OL.Row(1000, 1000)), OL.as_layout(OL.Col(1000, 1000))),
        ("transpose 999x1001", L.as_layout(L.Row(999, 1001)), L.as_layout(L.Col(999, 1001)),
         OL.as_layout(OL.Row(999, 1001)), OL.as_layout(OL.Col(999, 1001))),
        ("transpose 200x1000", L.as_layout(L.Row(200, 1000)), L.as_layout(L.Col(200, 1000)),
         OL.as_layout(OL.Row(200, 1000)), OL.as_layout(OL.Col(200, 1000))),
        ("transpose 192x320", L.as_layout(L.Row(192, 320)), L.as_layout(L.Col(192, 320)),
         OL.as_layout(OL.Row(192, 320)), OL.as_layout(OL.Col(192, 320))),
        # a whole matrix in antidiagonal order (Figure 7's GenP): 64x64 boxes
        # read in row order and written in antidiagonal order (or the
        # reverse), with ragged last boxes at 1000 and 130; at 63 the element
        # gather
        ("antidiagonal 1024^2", L.as_layout(L.Row(1024, 1024)), L.as_layout(L.GenP("antidiag", [1024, 1024])),
         OL.as_layout(OL.Row(1024, 1024)), OL.as_layout(OL.antidiag_genp(1024))),
        ("antidiagonal 1000^2", L.as_layout(L.Row(1000, 1000)), L.as_layout(L.GenP("antidiag", [1000, 1000])),
         OL.as_layout(OL.Row(1000, 1000)), OL.as_layout(OL.antidiag_genp(1000))),
        ("antidiagonal 130^2", L.as_layout(L.Row(130, 130)), L.as_layout(L.GenP("antidiag", [130, 130])),
         OL.as_layout(OL.Row(130, 130)), OL.as_layout(OL.antidiag_genp(130))),
        ("antidiagonal 63^2 (gather)", L.as_layout(L.Row(63, 63)), L.as_layout(L.GenP("antidiag", [63, 63])),
         OL.as_layout(OL.Row(63, 63)), OL.as_layout(OL.antidiag_genp(63))),
        # 3-D bricks (the stencil data layout of Section V): small ragged bricks and 8^3 bricks
        ("3-D bricks 2x5x3 of 6x10x12", L.as_layout(L.Row(6, 10, 12)), L.TileOrderBy(L.Row(3, 2, 4), L.Row(2, 5, 3)),
         OL.as_layout(OL.Row(6, 10, 12)), OL.TileOrderBy(OL.Row(3, 2, 4), OL.Row(2, 5, 3))),
        ("3-D bricks 8^3 of 128^3", L.as_layout(L.Row(128, 128, 128)),
         L.TileOrderBy(L.Row(16, 16, 16), L.Row(8, 8, 8)),
         OL.as_layout(OL.Row(128, 128, 128)), OL.TileOrderBy(OL.Row(16, 16, 16), OL.Row(8, 8, 8))),
    ]


def _random_piece(L, rng, r, c):
    """A random permutation piece over [r, c] (and its oracle twin): row- or
    column-major, reversal, an XOR swizzle (c a power of two), Morton order
    (powers of two) or the antidiagonal order (square)."""
    pow2 = lambda x: x & (x - 1) == 0
    kinds = ["row", "col", "reverse"]
    if pow2(c) and c >= 2:
        kinds.append("xor")
    if pow2(r) and pow2(c):
        kinds.append("morton")
    if r == c:
        kinds.append("antidiag")
    k = kinds[rng.integers(len(kinds))]
    if k == "row":
        return L.Row(r, c), OL.Row(r, c)
    if k == "col":
        return L.Col(r, c), OL.Col(r, c)
    if k == "reverse":
        return L.GenP("reverse", [r, c]), OL.reverse_genp(r, c)
    if k == "xor":
        v = int(2 ** rng.integers(0, int(np.log2(c)) + 1))
        sh = int(rng.integers(1, 5))
        return L.GenP("xor_swizzle", [r, c], [v, sh]), OL.xor_swizzle_genp(r, c, v, sh)
    if k == "morton":
        return L.GenP("morton", [r, c]), OL.morton_genp(r, c)
    return L.GenP("antidiag", [r, r]), OL.antidiag_genp(r)


def _random_layout(L, rng, R, C, tiles):
    """A whole layout over [R, C]: one piece, or TileOrderBy over the given
    tile shapes (each level a random piece)."""
    if not tiles:
        lp, op = _random_piece(L, rng, R, C)
        return L.as_layout(lp), OL.as_layout(op)
    dims = [(R // int(np.prod([t[0] for t in tiles])), C // int(np.prod([t[1] for t in tiles])))] + tiles
    ps = [_random_piece(L, rng, a, b) for a, b in dims]
    return L.TileOrderBy(*[p[0] for p in ps]), OL.TileOrderBy(*[p[1] for p in ps])


def _random_remap_cases(L):
    """24 remaps between random layouts of one logical shape, from a fixed
    seed: shapes of 1 to 3 tile levels whose tiles are small powers of two or
    odd sizes, each level a random piece (row/column-major, reversal, XOR
    swizzle, Morton, antidiagonal), element sizes of 1, 2, 4 and 8 bytes."""
    rng = np.random.default_rng(8091)
    sizes = [1, 2, 3, 4, 5, 7, 8, 16, 32, 64]
    out = []
    while len(out) < 24:
        levels = int(rng.integers(0, 3))
        tiles = [(sizes[rng.integers(len(sizes))], sizes[rng.integers(len(sizes))]) for _ in range(levels)]
        outer = (int(rng.integers(1, 40)), int(rng.integers(1, 40)))
        if rng.integers(3) == 0:
            outer = (int(2 ** rng.integers(0, 6)),) * 2
        R = outer[0] * int(np.prod([t[0] for t in tiles]))
        C = outer[1] * int(np.prod([t[1] for t in tiles]))
        if R * C > (1 << 22) or R * C < 2:
            continue
        # the source side may tile differently from the destination
        tiles_b = tiles if rng.integers(2) else []
        ls, ols = _random_layout(L, rng, R, C, tiles)
        ld, old = _random_layout(L, rng, R, C, tiles_b)
        elem = int((1, 2, 4, 8)[rng.integers(4)])
        out.append((f"random {len(out)}: {R}x{C} tiles {tiles}/{tiles_b} {elem} B", ls, ld, ols, old, elem))
    return out


@pytest.mark.parametrize("i", range(24))
def test_remap_random_layouts(lego, i):
    """A remap between two seeded random layouts and back, every byte against
    the oracle."""
    import torch
    dev = need_gpu()
    name, ls, ld, ols, old, elem = _random_remap_cases(lego)[i]
    n = ols.size()
    src = {1: lambda: (S.int_tensor(n) % 251).to(torch.uint8), 2: lambda: S.tensor(n, "f16", seed=7),
           4: lambda: S.tensor(n, "f32", seed=7), 8: lambda: S.int_tensor(n, bits=64)}[elem]()
    say(f"remap {name} plan={lego.remap_plan(ls, ld, elem)['info']}")
    out = _run(lego, ls, ld, src, dev)
    exp = OR.remap(ols, old, bits(src))
    assert (bits(out) == exp).all(), name
    say(f"remap back {name} plan={lego.remap_plan(ld, ls, elem)['info']}")
    back = _run(lego, ld, ls, out, dev)
    assert (bits(back) == bits(src)).all(), name


def _random_expand_cases(L):
    """12 seeded ExpandBy remaps: a compact row- or column-major array of
    ragged 2-D or 3-D extents against a random tiled layout of the padded
    shape (tiles of 1 to 16 per axis, each level a random piece in 2-D)."""
    rng = np.random.default_rng(91)
    out = []
    while len(out) < 12:
        d = 2 if rng.integers(3) else 3
        tile = [int((1, 2, 3, 4, 5, 8, 16)[rng.integers(7)]) for _ in range(d)]
        n = [int(rng.integers(1, 90 if d == 2 else 30)) for _ in range(d)]
        ne = [-(-a // t) * t for a, t in zip(n, tile)]
        if ne == n:
            continue
        inner = ("Row", "Col")[rng.integers(2)]
        ls = L.ExpandBy(n, ne, L.as_layout(getattr(L, inner)(*ne)))
        ols = OL.ExpandBy(n, ne, OL.as_layout(getattr(OL, inner)(*ne)))
        if d == 2:
            ld, old = _random_layout(L, rng, ne[0], ne[1], [tuple(tile)])
        else:
            outer = [a // t for a, t in zip(ne, tile)]
            ld, old = L.TileOrderBy(L.Row(*outer), L.Row(*tile)), OL.TileOrderBy(OL.Row(*outer), OL.Row(*tile))
        elem = int((1, 2, 4, 8)[rng.integers(4)])
        out.append((f"expand {n} into {ne} tiles {tile} {elem} B", ls, ld, ols, old, elem))
    return out


def _random_box_cases(L):
    """8 seeded remaps between a whole matrix in antidiagonal order (Figure 7)
    and a row-major, column-major or tiled layout, at sizes from 64 to 700
    (the box path, ragged last boxes included)."""
    rng = np.random.default_rng(92)
    out = []
    while len(out) < 8:
        n = int(rng.integers(64, 700))
        tiles = [] if rng.integers(2) else [(t, t) for t in (1, 2, 4, 5, 7, 8) if n % t == 0][-1:]
        ls, ols = _random_layout(L, rng, n, n, tiles) if tiles else (
            (L.as_layout(L.Row(n, n)), OL.as_layout(OL.Row(n, n))) if rng.integers(2) else
            (L.as_layout(L.Col(n, n)), OL.as_layout(OL.Col(n, n))))
        ld, old = L.as_layout(L.GenP("antidiag", [n, n])), OL.as_layout(OL.antidiag_genp(n))
        elem = int((1, 2, 4, 8)[rng.integers(4)])
        out.append((f"antidiagonal {n}^2 tiles {tiles} {elem} B", ls, ld, ols, old, elem))
    return out


def _fill(n, elem):
    import torch
    return {1: lambda: (S.int_tensor(n) % 251).to(torch.uint8), 2: lambda: S.tensor(n, "f16", seed=7),
            4: lambda: S.tensor(n, "f32", seed=7), 8: lambda: S.int_tensor(n, bits=64)}[elem]()


@pytest.mark.parametrize("i", range(12))
def test_remap_random_expandby(lego, i):
    """Pad a compact array into a random tiled layout (padding must read
    back zero) and crop it back, every byte against the oracle."""
    import torch
    dev = need_gpu()
    name, ls, ld, ols, old, elem = _random_expand_cases(lego)[i]
    src = _fill(OR.phys_size(ols), elem)
    say(f"remap {name} plan={lego.remap_plan(ls, ld, elem)['info']}")
    d_pad = torch.full((OR.phys_size(old),), 1, dtype=src.dtype, device=dev)
    lego.remap(ls, ld, src.to(dev), d_pad)
    torch.cuda.synchronize()
    assert (bits(d_pad.cpu()) == OR.remap(ols, old, bits(src))).all(), name
    say(f"remap crop {name} plan={lego.remap_plan(ld, ls, elem)['info']}")
    d_back = torch.empty(src.numel(), dtype=src.dtype, device=dev)
    lego.remap(ld, ls, d_pad, d_back)
    torch.cuda.synchronize()
    assert (bits(d_back.cpu()) == bits(src)).all(), name


@pytest.mark.parametrize("i", range(8))
def test_remap_random_antidiagonal(lego, i):
    dev = need_gpu()
    name, ls, ld, ols, old, elem = _random_box_cases(lego)[i]
    src = _fill(ols.size(), elem)
    say(f"remap {name} plan={lego.remap_plan(ls, ld, elem)['info']}")
    out = _run(lego, ls, ld, src, dev)
    assert (bits(out) == OR.remap(ols, old, bits(src))).all(), name
    say(f"remap back {name} plan={lego.remap_plan(ld, ls, elem)['info']}")
    back = _run(lego, ld, ls, out, dev)
    assert (bits(back) == bits(src)).all(), name


def _expand_cases(L):
    """ExpandBy (Section III-D, Figure 9): compact arrays whose extents the
    tiles do not divide, against tiled layouts of the padded shape."""
    def pad(n, ne, inner_l, inner_o):
        return L.ExpandBy(n, ne, inner_l), OL.ExpandBy(n, ne, inner_o)
    out = []
    for n, ne, tl, to in (
            ([5, 7], [6, 8], L.TileOrderBy(L.Row(3, 2), L.Row(2, 4)), OL.TileOrderBy(OL.Row(3, 2), OL.Row(2, 4))),
            ([1000, 1000], [1024, 1024], L.TileOrderBy(L.Col(16, 16), L.Row(64, 64)),
             OL.TileOrderBy(OL.Col(16, 16), OL.Row(64, 64))),
            ([999, 1001], [1024, 1024], L.TileOrderBy(L.Col(16, 16), L.Row(64, 64)),
             OL.TileOrderBy(OL.Col(16, 16), OL.Row(64, 64))),
            ([100, 99, 101], [104, 104, 104], L.TileOrderBy(L.Row(13, 13, 13), L.Row(8, 8, 8)),
             OL.TileOrderBy(OL.Row(13, 13, 13), OL.Row(8, 8, 8)))):
        ls, os_ = pad(n, ne, L.as_layout(L.Row(*ne)), OL.as_layout(OL.Row(*ne)))
        out.append((f"pad {'x'.join(map(str, n))} into {'x'.join(map(str, ne))}", ls, tl, os_, to))
    return out


def test_remap_pad_crop_8000_in_8192_full(lego):
    """The measured size: an 8000 x 8000 fp32 array into a zero-padded
    8192 x 8192 blocked buffer (64 x 64 tiles, column-major tile order) and
    back, every element against the oracle (padding must read back zero)."""
    import torch
    dev = need_gpu()
    n, ne = 8000, 8192
    ls = lego.ExpandBy([n, n], [ne, ne], lego.as_layout(lego.Row(ne, ne)))
    ld = lego.TileOrderBy(lego.Col(ne // 64, ne // 64), lego.Row(64, 64))
    ols = OL.ExpandBy([n, n], [ne, ne], OL.as_layout(OL.Row(ne, ne)))
    old = OL.TileOrderBy(OL.Col(ne // 64, ne // 64), OL.Row(64, 64))
    src = S.tensor(n * n, "f32", seed=S.SEED_SRC)
    say(f"remap pad 8000^2 into 8192^2 blocked plan={lego.remap_plan(ls, ld, 4)['info']}")
    d_pad = torch.full((ne * ne,), 1.0, dtype=torch.float32, device=dev)
    lego.remap(ls, ld, src.to(dev), d_pad)
    torch.cuda.synchronize()
    assert (bits(d_pad.cpu()) == OR.remap(ols, old, bits(src))).all()
    say(f"remap crop 8192^2 blocked to 8000^2 plan={lego.remap_plan(ld, ls, 4)['info']}")
    d_back = torch.empty(n * n, dtype=torch.float32, device=dev)
    lego.remap(ld, ls, d_pad, d_back)
    torch.cuda.synchronize()
    assert torch.equal(d_back.cpu(), src)


@pytest.mark.parametrize("elem", ["f32", "f16", "i64", "u8"])
def test_remap_expandby_pad_and_crop(lego, elem):
    """Compact -> padded tiled buffer (zero padding) -> compact again."""
    import torch
    dev = need_gpu()
    for name, ls, ld, ols, old in _expand_cases(lego):
        ns, nd = OR.phys_size(ols), OR.phys_size(old)
        if elem == "i64":
            src = S.int_tensor(ns, bits=64)
        elif elem == "u8":
            src = (S.int_tensor(ns) % 251).to(torch.uint8)
        else:
            src = S.tensor(ns, elem, seed=7)
        say(f"remap {name} {elem} plan={lego.remap_plan(ls, ld, src.element_size())['info']}")
        d_src = src.to(dev)
        d_pad = torch.full((nd,), 1, dtype=src.dtype, device=dev)  # padding must come back zero
        lego.remap(ls, ld, d_src, d_pad)
        torch.cuda.synchronize()
        exp = OR.remap(ols, old, bits(src))
        assert (bits(d_pad.cpu()) == exp).all(), name
        say(f"remap crop {name} {elem} plan={lego.remap_plan(ld, ls, src.element_size())['info']}")
        d_back = torch.empty_like(d_src)
        lego.remap(ld, ls, d_pad, d_back)
        torch.cuda.synchronize()
        assert (bits(d_back.cpu()) == bits(src)).all(), name


@pytest.mark.parametrize("elem", ["f32", "f16", "i64", "u8"])
def test_remap_small_and_ragged(lego, elem):
    import torch
    dev = need_gpu()
    for name, ls, ld, ols, old in _small_cases(lego):
        n = ols.size()
        if elem == "i64":
            src = S.int_tensor(n, bits=64)
        elif elem == "u8":
            src = (S.int_tensor(n) % 251).to(torch.uint8)
        else:
            src = S.tensor(n, elem, seed=7)
        say(f"remap {name} {elem} plan={lego.remap_plan(ls, ld, src.element_size())['info']}")
        out = _run(lego, ls, ld, src, dev)
        exp = OR.remap(ols, old, bits(src))
        assert (bits(out) == exp).all(), name
        back = _run(lego, ld, ls, out, dev)
        assert (bits(back) == bits(src)).all(), name


def test_remap_errors(lego):
    import torch
    dev = need_gpu()
    a = torch.zeros(64, device=dev)
    b = torch.zeros(64, device=dev)
    r = lego.as_layout(lego.Row(8, 8))
    with pytest.raises(lego.LegoError) as e:
        lego.remap(r, lego.as_layout(lego.Row(4, 16)), a, b)
    assert e.value.status == "SIZE_MISMATCH"
    with pytest.raises(lego.LegoError) as e:
        lego.remap(r, r, a, a)
    assert e.value.status == "INVALID_ARG"


def test_binding_follows_torch_current_stream(lego):
    """The binding launches on torch's current stream: the default one and a
    side stream entered with torch.cuda.stream (then the result is ordered
    after that stream's earlier work)."""
    import torch
    dev = need_gpu()
    assert (lego._stream(None).value or 0) == torch.cuda.current_stream().cuda_stream
    side = torch.cuda.Stream()
    n = 1024
    row, col = lego.as_layout(lego.Row(n, n)), lego.as_layout(lego.Col(n, n))
    src = S.tensor(n * n, "f32", seed=S.SEED_SRC)
    with torch.cuda.stream(side):
        assert lego._stream(None).value == side.cuda_stream
        x = src.to(dev, non_blocking=False)
        y = torch.empty_like(x)
        lego.remap(row, col, x, y)
    side.synchronize()
    assert (bits(y.cpu()) == bits(src).reshape(n, n).T.ravel()).all()
