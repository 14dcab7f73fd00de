"""User-defined GenPs from expression text, on the GPU: index maps and remaps
bit-exact against the oracle's independent evaluator of the same text, and a
GEMM whose LDS tiles use an expression-defined swizzle."""
import numpy as np
import pytest

import synth_inputs as S
from oracle import gemm as OG
from oracle import genexpr as GX
from oracle import layout as OL
from oracle import remap as OR
from tests import genp_exprs as GE
from tests.gpu_util import bits, need_gpu, say

pytestmark = pytest.mark.gpu


def _wavefront(L, G, n, t):
    """n x n matrix of t x t tiles: the tile grid in antidiagonal (wavefront)
    order written as an expression GenP, row-major inside each tile."""
    q = n // t
    if G is OL:
        return OL.GroupBy([n, n]).OrderBy(OL.RegP([q, t, q, t], [1, 3, 2, 4])).OrderBy(
            GX.expr_genp([q, q], GE.ANTIDIAG_APPLY, GE.ANTIDIAG_INV), OL.Row(t, t))
    return L.GroupBy([n, n]).OrderBy(L.RegP([q, t, q, t], [1, 3, 2, 4])).OrderBy(
        L.GenPExpr([q, q], GE.ANTIDIAG_APPLY, GE.ANTIDIAG_INV), L.Row(t, t))


def test_remap_wavefront_8192_full(lego):
    """The measured size: 8192^2 fp32 into 64 x 64 tiles in wavefront order
    (the expression GenP over the 128 x 128 tile grid) and back, every element
    against the oracle."""
    import torch
    dev = need_gpu()
    n = 8192
    ls, ld = lego.as_layout(lego.Row(n, n)), _wavefront(lego, None, n, 64)
    ols, old = OL.as_layout(OL.Row(n, n)), _wavefront(None, OL, n, 64)
    src = S.tensor(n * n, "f32", seed=S.SEED_SRC)
    say(f"remap wavefront 8192^2 plan={lego.remap_plan(ls, ld, 4)['info']}")
    d_src = src.to(dev)
    d_w = torch.empty_like(d_src)
    lego.remap(ls, ld, d_src, d_w)
    torch.cuda.synchronize()
    assert (d_w.cpu().numpy().view(np.uint32) == OR.remap(ols, old, src.numpy().view(np.uint32))).all()
    say(f"remap wavefront 8192^2 back plan={lego.remap_plan(ld, ls, 4)['info']}")
    d_back = torch.empty_like(d_src)
    lego.remap(ld, ls, d_w, d_back)
    torch.cuda.synchronize()
    assert torch.equal(d_back.cpu(), src)


SKEW_APPLY = "i1 * n0 + (i0 + i1) % n0"
SKEW_INV = ["(x % n0 + n0 - (x / n0) % n0) % n0", "x / n0"]


def _expr_cases(L):
    return [
        ("wavefront 2048^2 of 64x64 tiles", L.as_layout(L.Row(2048, 2048)), _wavefront(L, None, 2048, 64),
         OL.as_layout(OL.Row(2048, 2048)), _wavefront(None, OL, 2048, 64)),
        ("morton 8x8 tiles of 512^2", L.as_layout(L.Row(512, 512)),
         L.GroupBy([512, 512]).OrderBy(L.RegP([64, 8, 64, 8], [1, 3, 2, 4])).OrderBy(
             L.Row(64, 64), L.GenPExpr([8, 8], GE.MORTON8_APPLY, GE.MORTON8_INV)),
         OL.as_layout(OL.Row(512, 512)),
         OL.GroupBy([512, 512]).OrderBy(OL.RegP([64, 8, 64, 8], [1, 3, 2, 4])).OrderBy(
             OL.Row(64, 64), GX.expr_genp([8, 8], GE.MORTON8_APPLY, GE.MORTON8_INV))),
        # a skewed transpose of a 200 x 130 matrix, (i, j) -> j * 200 + (i + j) % 200:
        # no digit structure, ragged 64 x 64 boxes read in row order and
        # written in column order
        ("skewed transpose 200x130", L.as_layout(L.Row(200, 130)),
         L.as_layout(L.GenPExpr([200, 130], SKEW_APPLY, SKEW_INV)),
         OL.as_layout(OL.Row(200, 130)), OL.as_layout(GX.expr_genp([200, 130], SKEW_APPLY, SKEW_INV))),
    ]


@pytest.mark.parametrize("elem", ["f32", "f16"])
def test_remap_expression_layouts(lego, elem):
    import torch
    dev = need_gpu()
    for name, ls, ld, ols, old in _expr_cases(lego):
        n = OL.prod(ols.dims())
        src = S.tensor(n, elem, seed=5)
        say(f"remap {name} {elem} plan={lego.remap_plan(ls, ld, src.element_size())['info']}")
        d_src = src.to(dev)
        d_dst = torch.empty_like(d_src)
        lego.remap(ls, ld, d_src, d_dst)
        torch.cuda.synchronize()
        assert (bits(d_dst.cpu()) == OR.remap(ols, old, bits(src))).all(), name
        d_back = torch.empty_like(d_src)
        lego.remap(ld, ls, d_dst, d_back)
        torch.cuda.synchronize()
        assert (bits(d_back.cpu()) == bits(src)).all(), name


def test_index_maps_of_expression_layout(lego):
    import torch
    dev = need_gpu()
    lay = _wavefront(lego, None, 1024, 32)
    olay = _wavefront(None, OL, 1024, 32)
    n = 1024 * 1024
    say("index maps wavefront 1024^2 of 32x32 tiles")
    out = torch.empty(n, dtype=torch.int32, device=dev)
    lego.apply_all_device(lay, out)
    torch.cuda.synchronize()
    assert (out.cpu().numpy() == OL.apply_all(olay)).all()
    inv = torch.empty(n * 2, dtype=torch.int32, device=dev)
    lego.inv_all_device(lay, inv)
    torch.cuda.synchronize()
    assert (inv.cpu().numpy().reshape(n, 2) == OL.inv_all(olay)).all()


def test_gemm_with_expression_lds_swizzle(lego):
    """The LDS tiles of A and B use a swizzle given as expression text; the
    planner still proves the direct copies and vector fragment reads."""
    M = N = K = 1024
    a = S.tensor(M * K, "bf16", dist="normal", seed=S.SEED_A)
    b = S.tensor(K * N, "bf16", dist="normal", seed=S.SEED_B)
    sw = lego.as_layout(lego.GenPExpr([256, 64], GE.SWIZZLE64_APPLY, GE.SWIZZLE64_INV))
    kw = dict(lds_a=sw, lds_b=sw)
    plan = lego.gemm_plan(M, N, K, "bf16", **kw)
    say(f"gemm 1024 bf16 expression LDS plan={plan}")
    assert "direct-lds" in plan and "A:V8k sep svec frvec" in plan
    dev = need_gpu()
    import torch
    c = torch.full((M * N,), float("nan"), dtype=torch.float32, device=dev)
    lego.gemm(a.to(dev), b.to(dev), c, M, N, K, "bf16", **kw)
    torch.cuda.synchronize()
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(OL.Row(M, K)), OL.as_layout(OL.Col(K, N)), "bf16")
    ok, mre, fre = OG.check_tolerance(c.cpu().numpy().reshape(M, N), r)
    assert ok, (mre, fre)
