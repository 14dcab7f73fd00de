"""C ABI checks that need no GPU: exported symbols, error codes, host
evaluation of layouts against the oracle, lowering output."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import layout as OL

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "lego.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lego_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lego):
    lib = ctypes.CDLL(lego.library_path())
    names = _declared()
    assert len(names) >= 30
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    # and the binding exposes the same names
    assert set(names) <= set(lego.EXPORTED)


def test_version_and_last_error(lego):
    assert b"gfx950" in lego.lego_version()
    with pytest.raises(lego.LegoError):
        lego.RegP([2, 2], [1, 1])
    assert lego.lego_last_error()


@pytest.mark.parametrize("call,status", [
    (lambda L: L.RegP([2, 3], [1, 1]), "NOT_PERMUTATION"),
    (lambda L: L.RegP([2, 0], [1, 2]), "INVALID_ARG"),
    (lambda L: L.RegP([2, 3], [1]), "INVALID_ARG"),
    # empty extents: every layout and GEMM dimension must be positive
    (lambda L: L.Row(0, 4), "INVALID_ARG"),
    (lambda L: L.GroupBy([4, 0]), "INVALID_ARG"),
    (lambda L: L.gemm_plan(0, 64, 64, "f16"), "INVALID_ARG"),
    (lambda L: L.gemm_plan(64, 64, 0, "bf16"), "INVALID_ARG"),
    (lambda L: L.GroupBy([4, 4]).OrderBy(L.Row(3, 5)), "SIZE_MISMATCH"),
    (lambda L: L.GenP("morton", [6, 8]), "INVALID_ARG"),
    (lambda L: L.GenP("xor_swizzle", [8, 24], [8, 1]), "INVALID_ARG"),
    (lambda L: L.GenP("antidiag", [3, 4]), "INVALID_ARG"),
    (lambda L: L.GenP(99, [3, 3]), "INVALID_ARG"),
    (lambda L: L.as_layout(L.Row(4, 4)).apply([4, 0]), "OUT_OF_RANGE"),
    (lambda L: L.as_layout(L.Row(4, 4)).inv(16), "OUT_OF_RANGE"),
    (lambda L: L.ExpandBy([5, 7], [6, 9], L.TileOrderBy(L.Row(3, 2), L.Row(2, 4))), "SIZE_MISMATCH"),
    (lambda L: L.gemm_plan(64, 64, 64, "f16", bm=64, bn=64, bk=32, wm=48, wn=32), "UNSUPPORTED"),
    (lambda L: L.gemm_plan(64, 64, 64, "f32"), "INVALID_ARG"),
    (lambda L: L.gemm_plan(256, 256, 256, "f16", a=L.as_layout(L.Row(128, 256))), "SIZE_MISMATCH"),
    (lambda L: L.remap_plan(L.as_layout(L.Row(4, 4)), L.as_layout(L.Row(2, 8)), 4), "SIZE_MISMATCH"),
    (lambda L: L.remap_plan(L.as_layout(L.Row(4, 4)), L.as_layout(L.Row(4, 4)), 3), "INVALID_ARG"),
    (lambda L: L.gemm_plan(64, 64, 64, "f16", a=L.ExpandBy([60, 64], [64, 64], L.as_layout(L.Row(64, 64)))),
     "UNSUPPORTED"),
    (lambda L: L.mfma_fragment_layout(7, 0), "INVALID_ARG"),
    # TileOrderBy levels must all have rank d; GroupBy tile levels equal rank
    (lambda L: L._tileorderby_d(2, L.Row(4, 4), L.Row(2, 2, 2)), "INVALID_ARG"),
    (lambda L: L._tileorderby_d(3, L.Row(4, 4), L.Row(2, 2)), "INVALID_ARG"),
    (lambda L: L.GroupByTiles([4, 4], [2, 0]), "INVALID_ARG"),
    # LDS stages: 3 x 64 KiB of a 256x256x64 tile exceed the 160 KiB LDS; 1 is
    # no ring; a register-staged plan (A in 2x4 blocks) has exactly two
    (lambda L: L.gemm_plan(1024, 1024, 1024, "bf16", stages=3), "UNSUPPORTED"),
    (lambda L: L.gemm_plan(1024, 1024, 1024, "bf16", stages=1), "UNSUPPORTED"),
    (lambda L: L.gemm_plan(1024, 1024, 1024, "bf16", stages=3, a=L.TileOrderBy(L.Row(512, 256), L.Row(2, 4))),
     "UNSUPPORTED"),
])
def test_error_codes(lego, call, status):
    with pytest.raises(lego.LegoError) as e:
        call(lego)
    assert e.value.status == status


def test_null_pointers_rejected(lego):
    out = ctypes.c_void_p()
    assert lego.lego_regp(2, None, None, ctypes.byref(out)) == -1
    assert lego.lego_apply(None, None, None) == -1
    assert lego.lego_remap(None, None, 4, None, None, None) == -1
    lego.lego_release(None)  # ignored


def _pairs(L):
    return [
        (L.GroupBy([6, 4]).OrderBy(L.RegP([2, 2], [2, 1]), L.GenP("reverse", [3, 2])),
         OL.GroupBy([6, 4], chain=[OL.OrderBy(OL.RegP([2, 2], [2, 1]), OL.reverse_genp(3, 2))])),
        (L.GroupBy([6, 6]).OrderBy(L.RegP([2, 3, 2, 3], [1, 3, 2, 4])).OrderBy(L.RegP([2, 2], [2, 1]),
                                                                             L.GenP("antidiag", [3, 3])),
         OL.GroupBy([6, 6]).OrderBy(OL.RegP([2, 3, 2, 3], [1, 3, 2, 4])).OrderBy(OL.RegP([2, 2], [2, 1]),
                                                                               OL.antidiag_genp(3))),
        (L.TileBy([3, 4], [2, 5]), OL.TileBy([3, 4], [2, 5])),
        (L.TileOrderBy(L.Col(3, 5), L.Row(7, 3)), OL.TileOrderBy(OL.Col(3, 5), OL.Row(7, 3))),
        (L.as_layout(L.GenP("morton", [16, 8])), OL.as_layout(OL.morton_genp(16, 8))),
        (L.as_layout(L.GenP("xor_swizzle", [32, 32], [4, 2])), OL.as_layout(OL.xor_swizzle_genp(32, 32, 4, 2))),
        (L.as_layout(L.GenP("antidiag", [9, 9])), OL.as_layout(OL.antidiag_genp(9))),
        (L.GroupBy([2, 2, 2, 2, 2]).OrderBy(L.RegP([2] * 5, [5, 2, 4, 3, 1])),
         OL.GroupBy([2, 2, 2, 2, 2]).OrderBy(OL.RegP([2] * 5, [5, 2, 4, 3, 1]))),
        (L.GroupBy([3, 3], [4, 4]).OrderBy(L.Row(12, 12)), OL.GroupBy([3, 3], [4, 4]).OrderBy(OL.Row(12, 12))),
        (L.GroupBy([12, 20]).OrderBy(L.RegP([3, 4, 4, 5], [2, 4, 1, 3])).OrderBy(L.Col(16, 15))
         .OrderBy(L.GenP("reverse", [10, 24])),
         OL.GroupBy([12, 20]).OrderBy(OL.RegP([3, 4, 4, 5], [2, 4, 1, 3])).OrderBy(OL.Col(16, 15))
         .OrderBy(OL.reverse_genp(10, 24))),
        (L.ExpandBy([5, 7], [6, 8], L.TileOrderBy(L.Row(3, 2), L.Row(2, 4))),
         OL.ExpandBy([5, 7], [6, 8], OL.TileOrderBy(OL.Row(3, 2), OL.Row(2, 4)))),
    ]


def test_host_apply_inv_match_oracle(lego):
    for lay, olay in _pairs(lego):
        dims = lay.dims()
        assert dims == list(olay.dims())
        n = int(np.prod(dims))
        for x in range(n):
            idx = OL.canon_unflatten(dims, x)
            f = lay.apply(idx)
            assert f == int(olay.apply(idx))
            if f >= 0:
                assert lay.inv(f) == [int(v) for v in olay.inv(f)]


def test_verify_bijective(lego):
    for lay, _ in _pairs(lego):
        assert lay.verify_bijective()
    with pytest.raises(lego.LegoError) as e:
        lego.as_layout(lego.Row(8192, 8192)).verify_bijective(max_points=1000)
    assert e.value.status == "INVALID_ARG"


def test_emit_shows_closed_form_and_op_counts(lego):
    txt = lego.TileOrderBy(lego.Col(128, 128), lego.Row(64, 64)).emit("apply")
    assert "ops: 8" in txt and "u32" in txt and "/" not in txt.split("\n", 1)[1].replace("//", "")
    txt = lego.as_layout(lego.GenP("antidiag", [6, 6])).emit("inv")
    assert "lego_isqrt" in txt


def test_fragment_layouts_match_isa_formulas(lego):
    fa = lego.mfma_fragment_layout(0, 0)
    fc = lego.mfma_fragment_layout(0, 2)
    for lane in range(64):
        for e in range(8):
            assert fa.apply([lane, e]) == (lane % 32) * 16 + 8 * (lane // 32) + e
        for r in range(16):
            row, col = divmod(fc.apply([lane, r]), 32)
            assert (row, col) == (8 * (r // 4) + 4 * (lane // 32) + r % 4, lane % 32)
    fa16 = lego.mfma_fragment_layout(1, 0)
    fc16 = lego.mfma_fragment_layout(1, 2)
    for lane in range(64):
        for e in range(8):
            assert fa16.apply([lane, e]) == (lane % 16) * 32 + 8 * (lane // 16) + e
        for r in range(4):
            assert divmod(fc16.apply([lane, r]), 16) == (4 * (lane // 16) + r, lane % 16)


def test_plans_choose_expected_paths(lego):
    L = lego
    row = L.as_layout(L.Row(8192, 8192))
    blk = L.TileOrderBy(L.Col(128, 128), L.Row(64, 64))
    p = L.remap_plan(row, blk, 4)
    assert p["path"] == "direct" and p["run"] == 64 and p["vec"] == 4
    mz = L.as_layout(L.GenP("morton", [4096, 4096]))
    p = L.remap_plan(L.as_layout(L.Row(4096, 4096)), mz, 2)
    assert p["path"] == "lds" and p["vec"] == 8
    p = L.remap_plan(L.as_layout(L.Row(6, 6)), L.as_layout(L.GenP("antidiag", [6, 6])), 4)
    assert p["path"] == "gather"
    n = 4096
    row, ad = L.as_layout(L.Row(n, n)), L.as_layout(L.GenP("antidiag", [n, n]))
    p = L.remap_plan(row, ad, 4)
    assert p["path"] == "box" and p["tile"] == 4096 and "load rows sep (64 runs) store antidiags sep (127 runs)" in p["info"]
    p = L.remap_plan(ad, row, 4)
    assert p["path"] == "box" and "load antidiags sep (127 runs) store rows sep (64 runs)" in p["info"]
    # beyond the last-level cache: 128 x 128 boxes, the row side streaming
    n = 8192
    row, ad = L.as_layout(L.Row(n, n)), L.as_layout(L.GenP("antidiag", [n, n]))
    p = L.remap_plan(row, ad, 4)
    assert p["tile"] == 128 * 128 and "nt-loads" in p["info"] and "store antidiags sep" in p["info"]
    assert "nt-stores" in L.remap_plan(ad, row, 4)["info"]
    info = L.gemm_plan(8192, 8192, 8192, "bf16")
    assert "direct-lds spread fd2" in info and "A:V8k sep" in info and "frvec" in info
    assert "waves 2x2 wave 128x128" in info


def test_lds_plans_transfer_blocks_without_bank_conflicts(lego):
    """Transposing tiles move whole blocks (a thread's loads hold whole
    destination vectors, permuted in registers), and the planner's count of
    LDS bank passes over one tile finds none beyond the minimum for the
    transposes and the row -> Morton remap.  Morton -> row keeps scattered
    element writes: its destination vectors would need loads with gaps."""
    L = lego
    for n, eb in ((2048, 4), (4096, 4), (8192, 4), (4096, 2), (1024, 2)):
        info = L.remap_plan(L.as_layout(L.Row(n, n)), L.as_layout(L.Col(n, n)), eb)["info"]
        assert " block " in info and " bank-passes+0/0 " in info, (n, eb, info)
    row, mz = L.as_layout(L.Row(4096, 4096)), L.as_layout(L.GenP("morton", [4096, 4096]))
    info = L.remap_plan(row, mz, 2)["info"]
    assert " block 2x2 " in info and " bank-passes+0/0 " in info, info
    assert " scatter " in L.remap_plan(mz, row, 2)["info"]


def test_binding_checks_buffer_sizes_before_launch(lego):
    """The binding refuses buffers smaller than a layout's physical size
    (checked on the host, before any device call)."""
    import torch
    r = lego.as_layout(lego.Row(8, 8))
    e = lego.ExpandBy([5, 7], [8, 8], lego.as_layout(lego.Row(8, 8)))
    assert e.size() == 64 and e.phys_size() == 35 and r.phys_size() == 64
    with pytest.raises(lego.LegoError) as err:
        lego.remap(r, r, torch.zeros(63), torch.zeros(64))
    assert err.value.status == "SIZE_MISMATCH"
    with pytest.raises(lego.LegoError) as err:
        lego.remap(e, r, torch.zeros(35), torch.zeros(40))
    assert err.value.status == "SIZE_MISMATCH"
    with pytest.raises(lego.LegoError) as err:
        lego.remap(e, r, torch.zeros(35, dtype=torch.float16), torch.zeros(64))
    assert err.value.status == "INVALID_ARG"
    with pytest.raises(lego.LegoError) as err:
        lego.gemm(torch.zeros(64 * 64, dtype=torch.float16), torch.zeros(64 * 63, dtype=torch.float16),
                  torch.zeros(64 * 64), 64, 64, 64, "f16")
    assert err.value.status == "SIZE_MISMATCH"


def _all_points(lay):
    dims = lay.dims()
    return [list(p) for p in np.ndindex(*dims)]


def test_expression_genp_host_matches_oracle(lego):
    """GenPs from expression text evaluate on the host exactly as the oracle's
    independent evaluator of the same text, forward and inverse."""
    from oracle import genexpr as GX
    from tests import genp_exprs as GE
    cases = [([6, 6], GE.ANTIDIAG_APPLY, GE.ANTIDIAG_INV), ([8, 8], GE.MORTON8_APPLY, GE.MORTON8_INV),
             ([32, 64], GE.SWIZZLE64_APPLY, GE.SWIZZLE64_INV),
             ([3, 4, 5], "(i2 * n1 + i1) * n0 + i0", ["x % n0", "(x / n0) % n1", "x / (n0 * n1)"])]
    for dims, fwd, inv in cases:
        lay = lego.as_layout(lego.GenPExpr(dims, fwd, inv))
        ref = OL.as_layout(GX.expr_genp(dims, fwd, inv))
        for p in _all_points(lay):
            f = lay.apply(p)
            assert f == int(ref.apply(p))
            assert lay.inv(f) == [int(v) for v in ref.inv(f)]
    # in a chain, as a per-tile order (antidiagonal order of 2x2 tiles)
    lay = lego.GroupBy([6, 6]).OrderBy(lego.RegP([3, 2, 3, 2], [1, 3, 2, 4])).OrderBy(
        lego.GenPExpr([3, 3], GE.ANTIDIAG_APPLY, GE.ANTIDIAG_INV), lego.Row(2, 2))
    ref = OL.GroupBy([6, 6]).OrderBy(OL.RegP([3, 2, 3, 2], [1, 3, 2, 4])).OrderBy(OL.antidiag_genp(3), OL.Row(2, 2))
    for p in _all_points(lay):
        assert lay.apply(p) == int(ref.apply(p))


@pytest.mark.parametrize("fwd,inv,status", [
    ("i * n1 + j +", ["x / n1", "x % n1"], "INVALID_ARG"),         # syntax
    ("i * n1 + j", ["x / j", "x % n1"], "INVALID_ARG"),            # unknown name / non-constant divisor
    ("i * n1 + (j & 6)", ["x / n1", "x % n1"], "INVALID_ARG"),     # mask not 2^k - 1
    ("0", ["x / n1", "x % n1"], "NOT_BIJECTIVE"),                   # not a bijection
    ("i * n1 + j", ["x % n1", "x / n1"], "NOT_BIJECTIVE"),          # inverse does not invert
    ("i * n1 + j", ["x / n1"], "INVALID_ARG"),                      # one inverse per dimension
])
def test_expression_genp_errors(lego, fwd, inv, status):
    with pytest.raises(lego.LegoError) as e:
        lego.GenPExpr([4, 5], fwd, inv)
    assert e.value.status == status


@pytest.mark.parametrize("text,value", [
    ("1 + 2 * 3 << 1", 14), ("5 - 3 - 1", 1), ("2 ^ 3 & 1", 3), ("0 - 7 / 2", -3), ("-7 / 2", -4),
    ("-7 % 2", 1), ("1 < 2 == 1", 1), ("0 ? 5 : 1 ? 6 : 7", 6), ("isqrt(99)", 9), ("isqrt(100)", 10),
    ("max(3, min(9, 4))", 4), ("!0 + !5", 1), ("1 && 0 || 1", 1), ("3 >= 3 && 2 > 3", 0), ("6 != 6", 0),
])
def test_expression_language_host(lego, text, value):
    """The library's parser on the same hand-worked values as the oracle's:
    a shift of a 1009-point tile by the expression's value exposes it."""
    g = lego.as_layout(lego.GenPExpr([1009], f"i + ({text})", [f"x - ({text})"]))
    assert g.apply([0]) == value % 1009


def test_jit_uses_installed_compiler(tmp_path):
    """Kernels are compiled by the installed ROCm's compiler even in a process
    that imported a PyTorch wheel (which bundles an older compiler library
    under the same soname) first: the code objects name the compiler that
    /opt/rocm/llvm/bin/clang reports."""
    import subprocess
    import sys
    clang = "/opt/rocm/llvm/bin/clang"
    readelf = "/opt/rocm/llvm/bin/llvm-readelf"
    if not (os.path.exists(clang) and os.path.exists(readelf)):
        pytest.skip("no ROCm LLVM tools")
    want = subprocess.run([clang, "--version"], capture_output=True, text=True).stdout.splitlines()[0].strip()
    code = ("import torch\nimport paper_2505_08091_amd as L\n"
            "print(L.selftest_compile()[1].splitlines()[0])\n")
    env = dict(os.environ, LEGO_DUMP=str(tmp_path), PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "private namespace" in r.stdout, r.stdout
    objs = sorted(tmp_path.glob("*.co"))
    assert objs
    for o in objs[:3]:
        comment = subprocess.run([readelf, "-p", ".comment", str(o)], capture_output=True, text=True).stdout
        assert want in comment, (want, comment)


def test_one_hip_runtime_whatever_the_import_order():
    """Importing the package before torch leaves one HIP runtime and one HSA
    runtime in the process (torch's): with two, the second to open the GPU
    finds no device."""
    import subprocess
    import sys
    code = ("import paper_2505_08091_amd\nimport torch\n"
            "libs = {l.split()[-1] for l in open('/proc/self/maps') if 'amdhip64' in l or 'hsa-runtime64' in l}\n"
            "print(len({os.path.basename(p).split('.so')[0] for p in libs}), len(libs))\n")
    env = dict(os.environ, PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-c", "import os\n" + code], capture_output=True, text=True, env=env,
                       timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    kinds, files = map(int, r.stdout.split())
    assert kinds == files == 2, r.stdout


def test_retain_release_reference_counts(lego):
    """A retained handle outlives one release; the library drops it with the
    last one (composition holds its own references)."""
    import ctypes
    p = lego.Row(4, 4)
    lay = lego.as_layout(p)
    lib = lego._lib
    lib.lego_retain(p.h)          # two references
    lib.lego_release(p.h)         # one left: still valid
    d = (ctypes.c_int64 * 16)()
    r = ctypes.c_int()
    assert lib.lego_piece_dims(p.h, ctypes.byref(r), d) == 0 and list(d[:r.value]) == [4, 4]
    lib.lego_retain(None)         # NULL is ignored
    assert lay.apply([1, 2]) == 6


def test_fragment_layouts_select_instruction_on_host(lego):
    """frag_a/b/c given as the hardware's fragment layouts choose the MFMA
    instruction; mixed or foreign layouts are UNSUPPORTED; giving the default
    instruction's layouts generates the default kernel source."""
    f = [[lego.mfma_fragment_layout(i, op) for op in range(3)] for i in range(2)]
    p32 = lego.gemm_plan(1024, 1024, 1024, "bf16", frag_a=f[0][0], frag_b=f[0][1], frag_c=f[0][2])
    p16 = lego.gemm_plan(1024, 1024, 1024, "bf16", frag_c=f[1][2])
    assert "mfma 32x32x16" in p32 and "mfma 16x16x32" in p16
    assert lego.plan_source("gemm", M=1024, N=1024, K=1024, dtype="bf16", frag_a=f[0][0]) == \
        lego.plan_source("gemm", M=1024, N=1024, K=1024, dtype="bf16")
    for bad in (dict(frag_a=f[0][0], frag_c=f[1][2]), dict(frag_c=lego.as_layout(lego.Row(64, 16))),
                dict(frag_b=lego.as_layout(lego.Row(64, 8)))):
        with pytest.raises(lego.LegoError) as e:
            lego.gemm_plan(1024, 1024, 1024, "bf16", **bad)
        assert e.value.status == "UNSUPPORTED"


def test_gemm_argument_checks_before_any_device_work(lego):
    """Misaligned operands and a C that overlaps A or B are refused with
    INVALID_ARG before the library plans or launches anything (the pointers
    here are never dereferenced)."""
    import ctypes
    M = N = K = 256
    d = lego._desc(M, N, K, "f16")
    base = 1 << 20
    a, b, c = base, base + 2 * M * K, base + 4 * M * K
    cases = [(a + 8, b, c), (a, b + 2, c), (a, b, c + 2), (a, b, a + 1024), (a, b, b - 16)]
    for pa, pb, pc in cases:
        rc = lego._lib.lego_gemm(ctypes.byref(d), ctypes.c_void_p(pa), ctypes.c_void_p(pb), ctypes.c_void_p(pc), None)
        assert rc == -1, (pa, pb, pc, rc)


def test_index_map_output_alignment_checked(lego):
    """A device output that is not 16-byte aligned is refused before any launch."""
    import ctypes
    lay = lego.as_layout(lego.Row(8, 8))
    for f in (lego._lib.lego_apply_all_device, lego._lib.lego_inv_all_device):
        assert f(lay.h, 4, ctypes.c_void_p((1 << 20) + 4), None) == -1


def test_groupby_tiles_is_the_concatenated_logical_view(lego):
    """GroupBy over tile levels (Figure 3) has the levels' coordinates as its
    logical index: the same layout as a GroupBy over their concatenation, and
    chained with the same OrderBy it maps every point alike (Figure 6)."""
    g1 = lego.GroupByTiles([2, 3], [2, 3]).OrderBy(lego.RegP([2, 3, 2, 3], [1, 3, 2, 4]))
    g2 = lego.GroupBy([2, 3], [2, 3]).OrderBy(lego.RegP([2, 3, 2, 3], [1, 3, 2, 4]))
    o = OL.GroupBy([2, 3, 2, 3]).OrderBy(OL.RegP([2, 3, 2, 3], [1, 3, 2, 4]))
    assert g1.dims() == [2, 3, 2, 3]
    for x in range(36):
        idx = [int(v) for v in OL.canon_unflatten([2, 3, 2, 3], x)]
        assert g1.apply(idx) == g2.apply(idx) == int(o.apply(idx))


def test_gemm_stages_field(lego):
    """The descriptor's LDS stage count: 4 stages of a 256x256x32 tile fit
    (4 x 32 KiB); the plan reports what it uses, and 0 lets the planner choose."""
    assert " stages 4 " in lego.gemm_plan(1024, 1024, 1024, "bf16", bk=32, stages=4)
    assert " stages 2 " in lego.gemm_plan(1024, 1024, 1024, "bf16", bk=32, stages=2)
    assert " stages 2 " in lego.gemm_plan(1024, 1024, 1024, "bf16")
