"""Index maps on the GPU must equal the oracle bit for bit (every point)."""
import numpy as np
import pytest

from oracle import layout as OL
from tests.gpu_util import need_gpu, say

pytestmark = pytest.mark.gpu


def _cases(L):
    """(name, product layout, oracle layout) pairs."""
    return [
        ("C1 TileOrderBy(Row2x2,Row4x4,Row16x16)", L.TileOrderBy(L.Row(2, 2), L.Row(4, 4), L.Row(16, 16)),
         OL.TileOrderBy(OL.Row(2, 2), OL.Row(4, 4), OL.Row(16, 16))),
        ("C1 TileBy([2,2],[4,4],[16,16])", L.TileBy([2, 2], [4, 4], [16, 16]),
         OL.TileBy([2, 2], [4, 4], [16, 16])),
        ("Eq2 antidiag 6x6",
         L.GroupBy([6, 6]).OrderBy(L.RegP([2, 3, 2, 3], [1, 3, 2, 4])).OrderBy(L.RegP([2, 2], [2, 1]),
                                                                             L.GenP("antidiag", [3, 3])),
         OL.GroupBy([6, 6]).OrderBy(OL.RegP([2, 3, 2, 3], [1, 3, 2, 4])).OrderBy(OL.RegP([2, 2], [2, 1]),
                                                                               OL.antidiag_genp(3))),
        ("Fig2 reverse 6x4", L.GroupBy([6, 4]).OrderBy(L.RegP([2, 2], [2, 1]), L.GenP("reverse", [3, 2])),
         OL.GroupBy([6, 4], chain=[OL.OrderBy(OL.RegP([2, 2], [2, 1]), OL.reverse_genp(3, 2))])),
        ("Fig8 RegP 2^5", L.GroupBy([2, 2, 2, 2, 2]).OrderBy(L.RegP([2] * 5, [5, 2, 4, 3, 1])),
         OL.GroupBy([2, 2, 2, 2, 2]).OrderBy(OL.RegP([2] * 5, [5, 2, 4, 3, 1]))),
        ("Morton 64x64", L.as_layout(L.GenP("morton", [64, 64])), OL.as_layout(OL.morton_genp(64, 64))),
        ("Morton 32x128", L.as_layout(L.GenP("morton", [32, 128])), OL.as_layout(OL.morton_genp(32, 128))),
        ("XOR swizzle 256x64", L.as_layout(L.GenP("xor_swizzle", [256, 64], [8, 1])),
         OL.as_layout(OL.xor_swizzle_genp(256, 64, 8, 1))),
        ("antidiag 37x37", L.as_layout(L.GenP("antidiag", [37, 37])), OL.as_layout(OL.antidiag_genp(37))),
        ("ragged TileOrderBy 3x5 of 7x3", L.TileOrderBy(L.Col(3, 5), L.Row(7, 3)),
         OL.TileOrderBy(OL.Col(3, 5), OL.Row(7, 3))),
        ("grouped schedule 32x32 G=8", L.GroupBy([32, 32]).OrderBy(L.RegP([4, 8, 32], [1, 3, 2])),
         OL.GroupBy([32, 32]).OrderBy(OL.RegP([4, 8, 32], [1, 3, 2]))),
        ("chain of 3 OrderBys 12x20",
         L.GroupBy([12, 20]).OrderBy(L.RegP([3, 4, 4, 5], [2, 4, 1, 3])).OrderBy(L.Col(16, 15))
         .OrderBy(L.GenP("reverse", [10, 24])),
         OL.GroupBy([12, 20]).OrderBy(OL.RegP([3, 4, 4, 5], [2, 4, 1, 3])).OrderBy(OL.Col(16, 15))
         .OrderBy(OL.reverse_genp(10, 24))),
    ]


@pytest.mark.parametrize("idx_bytes", [4, 8])
def test_index_maps_small(lego, idx_bytes):
    import torch
    dev = need_gpu()
    for name, lay, olay in _cases(lego):
        n = olay.size()
        dt = torch.int32 if idx_bytes == 4 else torch.int64
        say(f"apply_all {name} n={n} idx_bytes={idx_bytes}")
        out = torch.full((n,), -7, dtype=dt, device=dev)
        lego.apply_all_device(lay, out)
        torch.cuda.synchronize()
        assert (out.cpu().numpy() == OL.apply_all(olay)).all(), name
        say(f"inv_all {name}")
        inv = torch.full((n, olay.dims().__len__()), -7, dtype=dt, device=dev)
        lego.inv_all_device(lay, inv)
        torch.cuda.synchronize()
        assert (inv.cpu().numpy() == OL.inv_all(olay)).all(), name


def _random_index_cases(L):
    """48 seeded random layouts: both sides of the random remap cases (one to
    three tile levels, each a row/column-major, reversed, XOR-swizzled, Morton
    or antidiagonal piece)."""
    from tests.test_gpu_remap import _random_remap_cases
    out = []
    for name, ls, ld, ols, old, _ in _random_remap_cases(L):
        out += [(name + " src", ls, ols), (name + " dst", ld, old)]
    return out


@pytest.mark.parametrize("idx_bytes", [4, 8])
def test_index_maps_random(lego, idx_bytes):
    import torch
    dev = need_gpu()
    dt = torch.int32 if idx_bytes == 4 else torch.int64
    for name, lay, olay in _random_index_cases(lego):
        n = olay.size()
        say(f"apply_all/inv_all {name} n={n} idx_bytes={idx_bytes}")
        out = torch.full((n,), -7, dtype=dt, device=dev)
        lego.apply_all_device(lay, out)
        inv = torch.full((n, len(olay.dims())), -7, dtype=dt, device=dev)
        lego.inv_all_device(lay, inv)
        torch.cuda.synchronize()
        assert (out.cpu().numpy() == OL.apply_all(olay)).all(), name
        assert (inv.cpu().numpy() == OL.inv_all(olay)).all(), name


def test_index_map_c2_full_size(lego):
    """The 8192^2 blocked layout on all 2^26 points (bit-exact)."""
    import torch
    dev = need_gpu()
    lay = lego.TileOrderBy(lego.Col(128, 128), lego.Row(64, 64))
    olay = OL.TileOrderBy(OL.Col(128, 128), OL.Row(64, 64))
    n = 8192 * 8192
    say("apply_all C2 blocked 8192^2")
    out = torch.empty(n, dtype=torch.int32, device=dev)
    lego.apply_all_device(lay, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    r = np.arange(n, dtype=np.int64) >> 13
    c = np.arange(n, dtype=np.int64) & 8191
    exp = ((c // 64) * 128 + r // 64) * 4096 + (r % 64) * 64 + c % 64  # closed form, pinned to the oracle
    assert (got == exp).all()
    # and the oracle itself on a sample of points
    idx = np.random.default_rng(0).integers(0, n, 100000)
    assert (got[idx] == np.asarray(olay.apply([idx >> 13, idx & 8191]))).all()
    say("inv_all C2 blocked 8192^2")
    inv = torch.empty((n, 2), dtype=torch.int32, device=dev)
    lego.inv_all_device(lay, inv)
    torch.cuda.synchronize()
    inv = inv.cpu().numpy()
    assert (inv[got, 0] == r).all() and (inv[got, 1] == c).all()


def test_expandby_apply_device(lego):
    """ExpandBy apply with the -1 sentinel (Figure 9) on the GPU."""
    import torch
    dev = need_gpu()
    g = lego.TileOrderBy(lego.Row(3, 2), lego.Row(2, 4))
    e = lego.ExpandBy([5, 7], [6, 8], g)
    og = OL.TileOrderBy(OL.Row(3, 2), OL.Row(2, 4))
    oe = OL.ExpandBy([5, 7], [6, 8], og)
    say("apply_all ExpandBy 5x7 in 6x8")
    out = torch.empty(48, dtype=torch.int64, device=dev)
    lego.apply_all_device(e, out)
    torch.cuda.synchronize()
    exp = np.array([oe.apply([i, j]) for i in range(6) for j in range(8)])
    assert (out.cpu().numpy() == exp).all()
