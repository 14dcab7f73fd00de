"""GEMM on the gfx950 matrix cores against the fp64 oracle.

Tolerance (fp16/bf16 inputs, fp32 accumulation, fp32 C): per element
|C - R| / max(|R|, ||R||_F / sqrt(MN)) <= 2e-2 and ||C - R||_F / ||R||_F <= 1e-3.
Small-integer inputs make every partial sum exact in fp32, so that case must
match the oracle bit for bit.
"""
import numpy as np
import pytest

import synth_inputs as S
from oracle import gemm as OG
from oracle import layout as OL
from oracle import remap as OR
from tests.gpu_util import bits, need_gpu, say

pytestmark = pytest.mark.gpu


def _run(lego, a_buf, b_buf, M, N, K, dtype, **kw):
    import torch
    dev = need_gpu()
    c = torch.full((M * N,), float("nan"), dtype=torch.float32, device=dev)
    lego.gemm(a_buf.to(dev), b_buf.to(dev), c, M, N, K, dtype, **kw)
    torch.cuda.synchronize()
    return c.cpu().numpy()


def _logical_c(c_flat, olc, rows=None):
    return OG.logical_matrix(c_flat.view(np.float32), olc, "f32", rows)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_gemm_c1_128(lego, dtype):
    """128^3 with 64x64 workgroup tiles of 16x16 wave tiles (16x16x32 MFMA)."""
    M = N = K = 128
    a = S.tensor(M * K, dtype, seed=S.SEED_A)
    b = S.tensor(K * N, dtype, seed=S.SEED_B)
    kw = dict(bm=64, bn=64, bk=32, wm=16, wn=16)
    say(f"gemm C1 {dtype} plan={lego.gemm_plan(M, N, K, dtype, **kw)}")
    c = _run(lego, a, b, M, N, K, dtype, **kw)
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(OL.Row(M, K)), OL.as_layout(OL.Col(K, N)), dtype)
    ok, mre, fre = OG.check_tolerance(c.reshape(M, N), r)
    assert ok, (mre, fre)


def test_gemm_c3_1024_f16(lego):
    """1024^3 fp16, A Row, B Col, 128x128x32 tiles, 64x64 wave tiles, grouped order."""
    M = N = K = 1024
    a = S.tensor(M * K, "f16", seed=S.SEED_A)
    b = S.tensor(K * N, "f16", seed=S.SEED_B)
    kw = dict(bm=128, bn=128, bk=32, wm=64, wn=64, group_m=8)
    say(f"gemm C3 plan={lego.gemm_plan(M, N, K, 'f16', **kw)}")
    c = _run(lego, a, b, M, N, K, "f16", **kw)
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(OL.Row(M, K)), OL.as_layout(OL.Col(K, N)), "f16")
    ok, mre, fre = OG.check_tolerance(c.reshape(M, N), r)
    assert ok, (mre, fre)


def test_gemm_exact_small_integers(lego):
    """Inputs in {-2..2}: the fp32 result is exact, so it must equal the oracle."""
    M, N, K = 512, 768, 1024
    a = S.tensor(M * K, "bf16", dist="smallint", seed=11)
    b = S.tensor(K * N, "bf16", dist="smallint", seed=12)
    say("gemm exact small-int 512x768x1024 bf16")
    c = _run(lego, a, b, M, N, K, "bf16")
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(OL.Row(M, K)), OL.as_layout(OL.Col(K, N)), "bf16")
    assert (c.reshape(M, N) == r).all()


def test_gemm_layout_variants(lego):
    """The four Row/Col variants of A and B (Section V-A) and a column-major C."""
    M, N, K = 256, 512, 384
    a = S.tensor(M * K, "f16", seed=S.SEED_A)
    b = S.tensor(K * N, "f16", seed=S.SEED_B)
    for la_name in ("Row", "Col"):
        for lb_name in ("Row", "Col"):
            la = getattr(lego, la_name)(M, K)
            lb = getattr(lego, lb_name)(K, N)
            ola = getattr(OL, la_name)(M, K)
            olb = getattr(OL, lb_name)(K, N)
            lc = lego.as_layout(lego.Col(M, N))
            kw = dict(a=lego.as_layout(la), b=lego.as_layout(lb), c=lc, bm=128, bn=128, bk=64, wm=64, wn=64)
            say(f"gemm A {la_name} B {lb_name} C Col plan={lego.gemm_plan(M, N, K, 'f16', **kw)}")
            c = _run(lego, a, b, M, N, K, "f16", **kw)
            r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(ola), OL.as_layout(olb), "f16")
            got = _logical_c(c, OL.as_layout(OL.Col(M, N)))
            ok, mre, fre = OG.check_tolerance(got, r)
            assert ok, (la_name, lb_name, mre, fre)


@pytest.mark.parametrize("instr", [0, 1])
def test_gemm_fragment_layouts_select_the_instruction(lego, instr):
    """The MFMA fragment layouts given as layouts (frag_a/b/c) pick the
    instruction: 32x32x16 (0) or 16x16x32 (1), on a 1024x768x512 bf16 GEMM."""
    M, N, K = 1024, 768, 512
    a = S.tensor(M * K, "bf16", dist="normal", seed=S.SEED_A)
    b = S.tensor(K * N, "bf16", dist="normal", seed=S.SEED_B)
    kw = dict(frag_a=lego.mfma_fragment_layout(instr, 0), frag_b=lego.mfma_fragment_layout(instr, 1),
              frag_c=lego.mfma_fragment_layout(instr, 2))
    plan = lego.gemm_plan(M, N, K, "bf16", **kw)
    say(f"gemm fragments instr {instr} plan={plan}")
    assert ("mfma 32x32x16" if instr == 0 else "mfma 16x16x32") in plan
    c = _run(lego, a, b, M, N, K, "bf16", **kw).reshape(M, N)
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(OL.Row(M, K)), OL.as_layout(OL.Col(K, N)),
                "bf16")
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


@pytest.mark.parametrize("staged,wn", [(False, 128), (True, 128), (False, 64), (True, 64)])
def test_gemm_wave_tiles(lego, staged, wn):
    """256x256 workgroup tiles with 128x128 wave tiles (256 accumulators, one
    wave per SIMD, the default) and with 128x64 wave tiles (two waves per
    SIMD): direct copies spread over the last substep with fragments read two
    substeps ahead, and, with A in 2x4 blocks, the register-staged rolling
    pipeline; 1024x512x1024 bf16 against the oracle."""
    M, N, K = 1024, 512, 1024
    a = S.tensor(M * K, "bf16", dist="normal", seed=S.SEED_A)
    b = S.tensor(K * N, "bf16", dist="normal", seed=S.SEED_B)
    kw = dict(bm=256, bn=256, bk=64, wm=128, wn=wn)
    ola = OL.as_layout(OL.Row(M, K))
    if staged:
        kw["a"] = lego.TileOrderBy(lego.Row(M // 2, K // 4), lego.Row(2, 4))
        ola = OL.TileOrderBy(OL.Row(M // 2, K // 4), OL.Row(2, 4))
    plan = lego.gemm_plan(M, N, K, "bf16", **kw)
    say(f"gemm wave tiles 128x{wn} staged={staged} plan={plan}")
    assert ("staged" in plan) == staged and f"wave 128x{wn}" in plan
    assert staged or "spread fd2" in plan
    c = _run(lego, a, b, M, N, K, "bf16", **kw).reshape(M, N)
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), ola, OL.as_layout(OL.Col(K, N)), "bf16")
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


def _sched_cases(L, mt, nt):
    """Workgroup schedules given as layouts over the [Mt, Nt] tile grid: tile
    (tm, tn) is computed by workgroup sched.apply(tm, tn)."""
    return [("row-major tile order", L.as_layout(L.Row(mt, nt)), 0),
            ("row-major tile order, XCD remap", L.as_layout(L.Row(mt, nt)), 1),
            ("column-major tile order", L.as_layout(L.Col(mt, nt)), 1),
            ("groups of 4 tile rows, as a chain", L.GroupBy([mt, nt]).OrderBy(L.RegP([mt // 4, 4, nt], [1, 3, 2])), 1),
            ("Morton tile order", L.as_layout(L.GenP("morton", [mt, nt])), 1)]


def test_gemm_user_schedules(lego):
    """GEMMs whose workgroup order is a user-given layout (Section II's
    grouped order is one such layout) against the oracle: the schedule moves
    work between workgroups but never changes C."""
    M, N, K = 2048, 2048, 512
    a = S.tensor(M * K, "bf16", dist="normal", seed=S.SEED_A)
    b = S.tensor(K * N, "bf16", dist="normal", seed=S.SEED_B)
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(OL.Row(M, K)), OL.as_layout(OL.Col(K, N)),
                "bf16")
    for name, sched, xcd in _sched_cases(lego, M // 256, N // 256):
        say(f"gemm schedule {name} plan={lego.gemm_plan(M, N, K, 'bf16', sched=sched, xcd_remap=xcd)}")
        c = _run(lego, a, b, M, N, K, "bf16", sched=sched, xcd_remap=xcd).reshape(M, N)
        ok, mre, fre = OG.check_tolerance(c, r)
        assert ok, (name, mre, fre)


def test_gemm_fragment_probe_one_hot(lego):
    """A = e_(m,k), B = e_(k,n): C must be exactly 1 at (m, n) and 0 elsewhere,
    which pins the C/D fragment layout of the MFMA instruction."""
    import torch
    M = N = K = 64
    rng = np.random.default_rng(0)
    for _ in range(6):
        m, k, n = (int(x) for x in rng.integers(0, 64, 3))
        a = torch.zeros(M * K, dtype=torch.float16)
        b = torch.zeros(K * N, dtype=torch.float16)
        a[m * K + k] = 1.0
        b[n * K + k] = 1.0  # B column-major
        for kw in (dict(bm=64, bn=64, bk=32, wm=32, wn=32), dict(bm=64, bn=64, bk=32, wm=16, wn=16)):
            say(f"gemm one-hot m={m} k={k} n={n} {kw}")
            c = _run(lego, a, b, M, N, K, "f16", **kw).reshape(M, N)
            exp = np.zeros((M, N), dtype=np.float32)
            exp[m, n] = 1.0
            assert (c == exp).all(), (m, k, n, kw)


def test_gemm_c4_8192_bf16(lego):
    """8192^3 bf16 with the default 256x256x64 plan (the measured
    configuration): every output element against the fp64 oracle; C is
    pre-filled with NaN so a tile that is never stored shows."""
    M = N = K = 8192
    a = S.tensor(M * K, "bf16", dist="normal", seed=S.SEED_A)
    b = S.tensor(K * N, "bf16", dist="normal", seed=S.SEED_B)
    say(f"gemm C4 plan={lego.gemm_plan(M, N, K, 'bf16')}")
    c = _run(lego, a, b, M, N, K, "bf16").reshape(M, N)
    assert np.isfinite(c).all()
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(OL.Row(M, K)), OL.as_layout(OL.Col(K, N)),
                "bf16")
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


def test_gemm_c5_morton_a(lego):
    """4096^3 fp16 with A stored in Morton order and B row-major.  The Morton
    buffer is made by the oracle's remap from the logical row-major values
    (and the device remap must produce the same bytes); every output element
    is checked against the fp64 oracle reading A through the Morton layout."""
    import torch
    M = N = K = 4096
    a_log = S.tensor(M * K, "f16", seed=S.SEED_A)  # logical row-major values
    b = S.tensor(K * N, "f16", seed=S.SEED_B)
    omz = OL.as_layout(OL.morton_genp(M, K))
    a_mz_bits = OR.remap(OL.as_layout(OL.Row(M, K)), omz, S.as_numpy_bits(a_log))
    a_mz = torch.from_numpy(a_mz_bits.view(np.float16).copy())
    mz = lego.as_layout(lego.GenP("morton", [M, K]))
    row = lego.as_layout(lego.Row(M, K))
    dev = need_gpu()
    say("remap 4096^2 f16 row->morton for the C5 operand")
    d_mz = torch.empty(M * K, dtype=torch.float16, device=dev)
    lego.remap(row, mz, a_log.to(dev), d_mz)
    torch.cuda.synchronize()
    assert (bits(d_mz.cpu()) == a_mz_bits).all()
    kw = dict(a=mz, b=lego.as_layout(lego.Row(K, N)))
    say(f"gemm C5 plan={lego.gemm_plan(M, N, K, 'f16', **kw)}")
    c = _run(lego, a_mz, b, M, N, K, "f16", **kw).reshape(M, N)
    assert np.isfinite(c).all()
    r = OG.gemm(a_mz_bits, S.as_numpy_bits(b), omz, OL.as_layout(OL.Row(K, N)), "f16")
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


def _morton_direct_cases(L):
    """Morton-order A copied directly into LDS (each 2 x 4 Z block in one
    slot).  With an even number of MFMA blocks per wave along m, blocks 2m
    and 2m+1 take the even and odd rows of a band and a lane reads both rows
    of its blocks (`frzpair`: the C rows follow the same order); otherwise a
    lane reads its row as dword pairs (`frdw`).  bf16 with column-major B,
    smaller tiles with row-major B (the transposing read beside it), 32-deep
    k-steps, a workgroup walking several tiles, and one-block-high wave tiles."""
    return [
        dict(M=1024, N=1024, K=1024, dtype="bf16", bl="Col", mode="frzpair"),
        dict(M=1024, N=512, K=2048, dtype="f16", bl="Row", bm=128, bn=128, bk=64, wm=64, wn=64, mode="frzpair"),
        dict(M=512, N=512, K=512, dtype="f16", bl="Col", bm=128, bn=128, bk=32, wm=64, wn=64, mode="frzpair"),
        dict(M=1024, N=1024, K=512, dtype="f16", bl="Row", max_workgroups=5, mode="frzpair"),
        dict(M=512, N=512, K=512, dtype="bf16", bl="Col", bm=64, bn=128, bk=64, wm=32, wn=64, mode="frdw"),
    ]


def _morton_direct_kw(L, case):
    kw = {k: v for k, v in case.items() if k not in ("bl", "mode")}
    kw["a"] = L.as_layout(L.GenP("morton", [case["M"], case["K"]]))
    kw["b"] = L.as_layout(getattr(L, case["bl"])(case["K"], case["N"]))
    return kw


@pytest.mark.parametrize("i", range(5))
def test_gemm_morton_a_direct(lego, i):
    """Morton-A GEMMs on the direct-copy path with dword fragment reads,
    every output element against the fp64 oracle reading A through its
    Morton layout (the A buffer made by the oracle's remap)."""
    import torch
    case = _morton_direct_cases(lego)[i]
    kw = _morton_direct_kw(lego, case)
    M, N, K, dt = kw.pop("M"), kw.pop("N"), kw.pop("K"), kw.pop("dtype")
    a_log = S.tensor(M * K, dt, seed=S.SEED_A)
    b = S.tensor(K * N, dt, seed=S.SEED_B)
    omz = OL.as_layout(OL.morton_genp(M, K))
    a_mz_bits = OR.remap(OL.as_layout(OL.Row(M, K)), omz, S.as_numpy_bits(a_log))
    a_mz = torch.from_numpy(a_mz_bits.view(np.int16).copy()).view(a_log.dtype)
    plan = lego.gemm_plan(M, N, K, dt, **{k: v for k, v in kw.items() if k != "max_workgroups"})
    say(f"gemm Morton-A direct {case} plan={plan}")
    assert f" {case['mode']} " in plan and "direct-lds" in plan, plan
    c = _run(lego, a_mz, b, M, N, K, dt, **kw).reshape(M, N)
    assert np.isfinite(c).all()
    r = OG.gemm(a_mz_bits, S.as_numpy_bits(b), omz, OL.as_layout(getattr(OL, case["bl"])(K, N)), dt)
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


@pytest.mark.parametrize("la_name,lb_name", [("Row", "Row"), ("Row", "Col"), ("Col", "Row"), ("Col", "Col")])
def test_gemm_operand_layouts_4096(lego, la_name, lb_name):
    """The four Row/Col operand variants of Section V-A at 4096^3 fp16 with
    the default plan: every output element against the oracle."""
    M = N = K = 4096
    a = S.tensor(M * K, "f16", seed=S.SEED_A)
    b = S.tensor(K * N, "f16", seed=S.SEED_B)
    kw = dict(a=lego.as_layout(getattr(lego, la_name)(M, K)), b=lego.as_layout(getattr(lego, lb_name)(K, N)))
    say(f"gemm 4096 A {la_name} B {lb_name} plan={lego.gemm_plan(M, N, K, 'f16', **kw)}")
    c = _run(lego, a, b, M, N, K, "f16", **kw).reshape(M, N)
    assert np.isfinite(c).all()
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(getattr(OL, la_name)(M, K)),
                OL.as_layout(getattr(OL, lb_name)(K, N)), "f16")
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


@pytest.mark.parametrize("la_name,lb_name", [("Row", "Row"), ("Row", "Col"), ("Col", "Row"), ("Col", "Col")])
def test_gemm_operand_layouts_8192(lego, la_name, lb_name):
    """The four Row/Col operand variants at the measured 8192^3 fp16, default
    plan: every output element against the fp64 oracle."""
    M = N = K = 8192
    a = S.tensor(M * K, "f16", seed=S.SEED_A)
    b = S.tensor(K * N, "f16", seed=S.SEED_B)
    kw = dict(a=lego.as_layout(getattr(lego, la_name)(M, K)), b=lego.as_layout(getattr(lego, lb_name)(K, N)))
    say(f"gemm 8192 A {la_name} B {lb_name} plan={lego.gemm_plan(M, N, K, 'f16', **kw)}")
    c = _run(lego, a, b, M, N, K, "f16", **kw).reshape(M, N)
    assert np.isfinite(c).all()
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(getattr(OL, la_name)(M, K)),
                OL.as_layout(getattr(OL, lb_name)(K, N)), "f16")
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


def test_gemm_ragged_8000_bf16_full(lego):
    """The measured partial-tile GEMM, 8000^3 bf16 with 256-wide tiles that
    overhang the matrices: every output element against the fp64 oracle."""
    M = N = K = 8000
    a = S.tensor(M * K, "bf16", dist="normal", seed=S.SEED_A)
    b = S.tensor(K * N, "bf16", dist="normal", seed=S.SEED_B)
    say(f"gemm ragged 8000^3 plan={lego.gemm_plan(M, N, K, 'bf16')}")
    c = _run(lego, a, b, M, N, K, "bf16").reshape(M, N)
    assert np.isfinite(c).all()
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(OL.Row(M, K)), OL.as_layout(OL.Col(K, N)),
                "bf16")
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


def test_gemm_errors(lego):
    import torch
    dev = need_gpu()
    a = torch.zeros(100 * 64, dtype=torch.float16, device=dev)
    c = torch.zeros(100 * 64, dtype=torch.float32, device=dev)
    with pytest.raises(lego.LegoError) as e:
        lego.gemm(a, a, c, 64, 64, 64, "f16", wm=48)  # wave tile not a multiple of the MFMA block
    assert e.value.status == "UNSUPPORTED"
    with pytest.raises(lego.LegoError) as e:
        lego.gemm(a, a, c, 64, 64, 64, "f32")
    assert e.value.status == "INVALID_ARG"


@pytest.mark.parametrize("la_name,lb_name", [("Row", "Row"), ("Col", "Row"), ("Col", "Col")])
def test_gemm_mn_contiguous_operands_2048(lego, la_name, lb_name):
    """2048^3 fp16 with the default 256x256x64 plan for operands contiguous
    along m or n (read into fragments with the transposing LDS load), every
    output element against the oracle."""
    M = N = K = 2048
    a = S.tensor(M * K, "f16", seed=S.SEED_A)
    b = S.tensor(K * N, "f16", seed=S.SEED_B)
    kw = dict(a=lego.as_layout(getattr(lego, la_name)(M, K)), b=lego.as_layout(getattr(lego, lb_name)(K, N)))
    plan = lego.gemm_plan(M, N, K, "f16", **kw)
    say(f"gemm 2048 A {la_name} B {lb_name} plan={plan}")
    assert "frtr" in plan
    c = _run(lego, a, b, M, N, K, "f16", **kw).reshape(M, N)
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), OL.as_layout(getattr(OL, la_name)(M, K)),
                OL.as_layout(getattr(OL, lb_name)(K, N)), "f16")
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


def _ragged_cases(L):
    """Sizes the tiles do not divide (partial tiles, Section III-D): padded
    loads read zero, stores outside C are dropped; includes a ragged last
    group of the grouped schedule (9 tile rows, groups of 8), a K tail that
    is not a multiple of the 16-byte vector, and transposed-operand layouts."""
    return [
        dict(M=1000, N=1000, K=1000, dtype="bf16"),
        dict(M=513, N=257, K=320, dtype="f16"),
        dict(M=100, N=200, K=64, dtype="f16"),
        dict(M=64, N=64, K=36, dtype="f16"),
        dict(M=2100, N=300, K=136, dtype="bf16"),
        dict(M=1000, N=1000, K=1000, dtype="f16", a=L.as_layout(L.Col(1000, 1000)), b=L.as_layout(L.Row(1000, 1000))),
        dict(M=77, N=1, K=5, dtype="f16"),
        dict(M=1, N=1, K=1, dtype="bf16"),
        # register-staged loads (the rolling pipeline) with partial tiles: A in
        # 2x4 blocks (4-element k runs), then also B in 4x8 column-major blocks
        # (element loads)
        dict(M=1002, N=520, K=1000, dtype="bf16", a=L.TileOrderBy(L.Row(501, 250), L.Row(2, 4)),
             oa=OL.TileOrderBy(OL.Row(501, 250), OL.Row(2, 4))),
        dict(M=1002, N=520, K=1000, dtype="f16", a=L.TileOrderBy(L.Row(501, 250), L.Row(2, 4)),
             b=L.TileOrderBy(L.Row(250, 65), L.Col(4, 8)),
             oa=OL.TileOrderBy(OL.Row(501, 250), OL.Row(2, 4)), ob=OL.TileOrderBy(OL.Row(250, 65), OL.Col(4, 8))),
        # M or N below one wave tile: whole MFMA blocks hold no element of C,
        # with transposing fragment reads of B (N = 56 of 128, A Morton) and
        # of A (M = 40 of 128, column-major)
        dict(M=512, N=56, K=512, dtype="bf16", a=L.as_layout(L.GenP("morton", [512, 512])),
             b=L.as_layout(L.Row(512, 56)), bm=128, bn=256, bk=64, wm=64, wn=128,
             oa=OL.as_layout(OL.morton_genp(512, 512)), ob=OL.as_layout(OL.Row(512, 56))),
        dict(M=40, N=512, K=128, dtype="f16", a=L.as_layout(L.Col(40, 128)), b=L.as_layout(L.Col(128, 512)),
             bm=256, bn=256, bk=64, wm=128, wn=128, oa=OL.as_layout(OL.Col(40, 128)), ob=OL.as_layout(OL.Col(128, 512))),
    ]


@pytest.mark.parametrize("i", range(12))
def test_gemm_ragged_sizes(lego, i):
    """Every output element of a GEMM with partial tiles against the oracle;
    C is pre-filled with NaN so a dropped or misplaced store shows."""
    kw = dict(_ragged_cases(lego)[i])
    M, N, K, dtype = kw.pop("M"), kw.pop("N"), kw.pop("K"), kw.pop("dtype")
    oa, ob = kw.pop("oa", None), kw.pop("ob", None)
    a = S.tensor(M * K, dtype, seed=S.SEED_A)
    b = S.tensor(K * N, dtype, seed=S.SEED_B)
    say(f"gemm ragged {M}x{N}x{K} {dtype} plan={lego.gemm_plan(M, N, K, dtype, **kw)}")
    c = _run(lego, a, b, M, N, K, dtype, **kw).reshape(M, N)
    ola = oa if oa is not None else OL.as_layout(OL.Col(M, K)) if "a" in kw else OL.as_layout(OL.Row(M, K))
    olb = ob if ob is not None else OL.as_layout(OL.Row(K, N)) if "b" in kw else OL.as_layout(OL.Col(K, N))
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), ola, olb, dtype)
    assert np.isfinite(c).all()
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


def _random_cases(L):
    """36 GEMM configurations drawn from fixed seeds: fp16 or bf16; A
    row-major, column-major or in Morton order (power-of-two M and K), B row-
    or column-major; the default tiles or one of six smaller tile and wave
    shapes; ragged sizes unless A is in Morton order; and now and then a
    workgroup cap, so that workgroups walk several tiles.  Configurations the
    planner rejects are drawn again."""
    rng = np.random.default_rng(2505)
    tiles = [None, (128, 128, 64, 64, 64), (128, 128, 32, 64, 64), (64, 64, 32, 32, 32), (64, 128, 64, 32, 64),
             (256, 128, 64, 128, 64), (128, 256, 64, 64, 128)]
    out = []
    while len(out) < 24:
        dt = ("f16", "bf16")[rng.integers(2)]
        la, lb = ("Row", "Col", "Morton")[rng.integers(3)], ("Row", "Col")[rng.integers(2)]
        if la == "Morton":
            M, K = (int(x) for x in 2 ** rng.integers(6, 10, 2))
        else:
            M, K = (int(x) for x in rng.integers(1, 700, 2))
        N = int(rng.integers(1, 700))
        if rng.integers(2):  # whole tiles: the plan may walk tiles (persistent)
            N = 256 * int(rng.integers(1, 3))
            if la != "Morton":
                M, K = 256 * int(rng.integers(1, 3)), 256 * int(rng.integers(1, 3))
        kw = dict(M=M, N=N, K=K, dtype=dt)
        t = tiles[rng.integers(len(tiles))]
        if t:
            kw.update(bm=t[0], bn=t[1], bk=t[2], wm=t[3], wn=t[4])
        if la == "Morton":
            kw["a"], kw["oa"] = L.as_layout(L.GenP("morton", [M, K])), OL.as_layout(OL.morton_genp(M, K))
        else:
            kw["a"], kw["oa"] = L.as_layout(getattr(L, la)(M, K)), OL.as_layout(getattr(OL, la)(M, K))
        kw["b"], kw["ob"] = L.as_layout(getattr(L, lb)(K, N)), OL.as_layout(getattr(OL, lb)(K, N))
        try:
            L.gemm_plan(M, N, K, dt, **{k: v for k, v in kw.items() if k not in ("M", "N", "K", "dtype", "oa", "ob")})
        except L.LegoError:
            continue
        if rng.integers(3) == 0:
            kw["max_workgroups"] = int(rng.integers(1, 8))
        out.append(kw)
    # 12 more with explicit tiles, LDS layouts given as XOR swizzles of random
    # granule and stride, and a workgroup order given as a layout
    rng = np.random.default_rng(2506)
    while len(out) < 36:
        dt = ("f16", "bf16")[rng.integers(2)]
        la, lb = ("Row", "Col")[rng.integers(2)], ("Row", "Col")[rng.integers(2)]
        t = tiles[1 + rng.integers(len(tiles) - 1)]
        bm, bn, bk = t[0], t[1], t[2]
        M, N, K = bm * int(rng.integers(1, 4)), bn * int(rng.integers(1, 4)), bk * int(rng.integers(1, 5))
        kw = dict(M=M, N=N, K=K, dtype=dt, bm=bm, bn=bn, bk=bk, wm=t[3], wn=t[4])
        kw["a"], kw["oa"] = L.as_layout(getattr(L, la)(M, K)), OL.as_layout(getattr(OL, la)(M, K))
        kw["b"], kw["ob"] = L.as_layout(getattr(L, lb)(K, N)), OL.as_layout(getattr(OL, lb)(K, N))
        for side, rows in (("lds_a", bm), ("lds_b", bn)):
            if rng.integers(2):
                v = int((8, 16, 32)[rng.integers(3)])
                if v <= bk:
                    kw[side] = L.as_layout(L.GenP("xor_swizzle", [rows, bk], [v, int(rng.integers(1, 5))]))
        mt, nt = M // bm, N // bn
        sched = rng.integers(4)
        if sched == 1:
            kw["sched"] = L.as_layout(L.Col(mt, nt))
        elif sched == 2:
            kw["sched"] = L.as_layout(L.GenP("reverse", [mt, nt]))
        elif sched == 3 and mt & (mt - 1) == 0 and nt & (nt - 1) == 0:
            kw["sched"] = L.as_layout(L.GenP("morton", [mt, nt]))
        try:
            L.gemm_plan(M, N, K, dt, **{k: v for k, v in kw.items() if k not in ("M", "N", "K", "dtype", "oa", "ob")})
        except L.LegoError:
            continue
        out.append(kw)
    return out


@pytest.mark.parametrize("i", range(36))
def test_gemm_random_configs(lego, i):
    """Every output element of a seeded random GEMM configuration against the
    fp64 oracle (C pre-filled with NaN)."""
    kw = dict(_random_cases(lego)[i])
    M, N, K, dtype = kw.pop("M"), kw.pop("N"), kw.pop("K"), kw.pop("dtype")
    oa, ob = kw.pop("oa"), kw.pop("ob")
    a_log = S.tensor(M * K, dtype, seed=S.SEED_A)
    b_log = S.tensor(K * N, dtype, seed=S.SEED_B)
    # operands stored in their layouts by the oracle's remap of row-major values
    a_bits = OR.remap(OL.as_layout(OL.Row(M, K)), oa, S.as_numpy_bits(a_log))
    b_bits = OR.remap(OL.as_layout(OL.Row(K, N)), ob, S.as_numpy_bits(b_log))
    import torch
    a = torch.from_numpy(a_bits.view(np.int16).copy()).view(a_log.dtype)
    b = torch.from_numpy(b_bits.view(np.int16).copy()).view(b_log.dtype)
    say(f"gemm random {i}: {M}x{N}x{K} {dtype} plan={lego.gemm_plan(M, N, K, dtype, **{k: v for k, v in kw.items() if k != 'max_workgroups'})}")
    c = _run(lego, a, b, M, N, K, dtype, **kw).reshape(M, N)
    assert np.isfinite(c).all()
    r = OG.gemm(a_bits, b_bits, oa, ob, dtype)
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)


@pytest.mark.parametrize("layouts", ["row_col", "col_row"])
def test_gemm_operand_of_2gib(lego, layouts):
    """A 32768 x 32768 bf16 A operand (2 GiB: copies through 64-bit
    addresses, not the range-checked buffer loads), N = 256: two sampled rows
    of every 256-row tile row against the fp64 oracle.  The operands are made
    on the device by a seeded torch generator and the sampled rows read
    back as inputs of the check."""
    import torch
    dev = need_gpu()
    M, N, K = 32768, 256, 32768
    la, lb = ("Row", "Col") if layouts == "row_col" else ("Col", "Row")
    kw = dict(a=lego.as_layout(getattr(lego, la)(M, K)), b=lego.as_layout(getattr(lego, lb)(K, N)))
    plan = lego.gemm_plan(M, N, K, "bf16", **kw)
    say(f"gemm 2 GiB operand {layouts} plan={plan}")
    g = torch.Generator(device=dev)
    g.manual_seed(2505)
    a = torch.randn(M * K, generator=g, device=dev).to(torch.bfloat16)
    b = torch.randn(K * N, generator=g, device=dev).to(torch.bfloat16)
    c = torch.full((M * N,), float("nan"), dtype=torch.float32, device=dev)
    lego.gemm(a, b, c, M, N, K, "bf16", **kw)
    torch.cuda.synchronize()
    rows = np.sort(np.concatenate([np.arange(0, M, 256), np.arange(0, M, 256) + 255 - np.arange(M // 256) % 256]))
    ri = torch.from_numpy(rows).to(dev)
    if la == "Row":
        a_rows = a.view(M, K)[ri]
    else:
        a_rows = a.view(K, M)[:, ri].t().contiguous()
    a_bits = a_rows.view(torch.int16).cpu().numpy().view(np.uint16)  # the sampled rows, row-major
    b_bits = b.view(torch.int16).cpu().numpy().view(np.uint16)
    r = OG.gemm(a_bits, b_bits, OL.as_layout(OL.Row(rows.size, K)), OL.as_layout(getattr(OL, lb)(K, N)), "bf16")
    got = c.view(M, N)[ri].cpu().numpy()
    assert np.isfinite(got).all()
    ok, mre, fre = OG.check_tolerance(got, r)
    assert ok, (mre, fre)
    del a, b, c


def _persistent_cases(L):
    """GEMMs whose workgroups each walk several output tiles (the plan is
    persistent and max_workgroups is below the tile count), so the LDS ring
    chains from one tile into the next: uneven tile counts per workgroup,
    k-step counts that do not divide by the stage count (the ring's first
    stage alternates between tiles), four 32-deep stages, the transposing
    fragment reads, and a single workgroup doing everything (plans with
    partial tiles do not walk)."""
    return [
        dict(M=1024, N=512, K=1024, dtype="bf16", max_workgroups=3),
        dict(M=1024, N=768, K=320, dtype="f16", max_workgroups=5),
        dict(M=1024, N=512, K=1024, dtype="bf16", bk=32, stages=4, max_workgroups=3),
        dict(M=1024, N=512, K=1024, dtype="f16", a=L.as_layout(L.Col(1024, 1024)), b=L.as_layout(L.Row(1024, 512)),
             oa=OL.as_layout(OL.Col(1024, 1024)), ob=OL.as_layout(OL.Row(1024, 512)), max_workgroups=3),
        dict(M=1024, N=512, K=512, dtype="bf16", max_workgroups=1),
    ]


@pytest.mark.parametrize("i", range(5))
def test_gemm_persistent_tile_walk(lego, i):
    kw = dict(_persistent_cases(lego)[i])
    M, N, K, dtype = kw.pop("M"), kw.pop("N"), kw.pop("K"), kw.pop("dtype")
    oa = kw.pop("oa", OL.as_layout(OL.Row(M, K)))
    ob = kw.pop("ob", OL.as_layout(OL.Col(K, N)))
    a = S.tensor(M * K, dtype, dist="normal", seed=S.SEED_A)
    b = S.tensor(K * N, dtype, dist="normal", seed=S.SEED_B)
    plan = lego.gemm_plan(M, N, K, dtype, **kw)
    say(f"gemm persistent {M}x{N}x{K} {dtype} {kw.get('max_workgroups')} workgroups plan={plan}")
    assert "persistent" in plan
    c = _run(lego, a, b, M, N, K, dtype, **kw).reshape(M, N)
    assert np.isfinite(c).all()
    r = OG.gemm(S.as_numpy_bits(a), S.as_numpy_bits(b), oa, ob, dtype)
    ok, mre, fre = OG.check_tolerance(c, r)
    assert ok, (mre, fre)
