"""Checks on the gfx950 code objects the library generates (CPU only: hipRTC
cross-compiles, the ROCm disassembler reads the result).

The GEMM reads fragments of operands that are contiguous along m or n with
the transposing LDS load ds_read_b64_tr_b16, issued as inline assembly (the
compiler's own form of the load is ordered behind every direct global-to-LDS
copy in flight).  The compiler does not know when such a load completes: the
kernel itself waits for all LDS loads (s_waitcnt lgkmcnt(0)) before it uses a
fragment.  That is only sound if no instruction touches a load's destination
registers between the load and that wait - for instance a register copy that
packs the two 64-bit halves into the 128-bit MFMA operand.  These tests
disassemble every generated GEMM that uses the load and check that property
on every control-flow path.
"""
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"

_ADDR = re.compile(r"//\s*([0-9A-Fa-f]+):")
_FUNC = re.compile(r"^([0-9a-f]+) <([^>]+)>:")
_TARGET = re.compile(r"<([^+>]+)\+0x([0-9a-f]+)>")
_VRANGE = re.compile(r"\bv\[(\d+):(\d+)\]")
_VONE = re.compile(r"\bv(\d+)\b")


def parse(text):
    """Instructions of a disassembly as (address, mnemonic, operand text,
    branch target address or None), in address order."""
    funcs, out = {}, []
    for line in text.splitlines():
        m = _FUNC.match(line)
        if m:
            funcs[m.group(2)] = int(m.group(1), 16)
            continue
        m = _ADDR.search(line)
        if not m or not line.startswith("\t"):
            continue
        body = line.split("//")[0].strip()
        if not body:
            continue
        mnem, _, ops = body.partition(" ")
        tgt = None
        t = _TARGET.search(line)
        if t and (mnem.startswith("s_cbranch") or mnem == "s_branch"):
            tgt = funcs[t.group(1)] + int(t.group(2), 16)
        out.append((int(m.group(1), 16), mnem, ops, tgt))
    return out


def vregs(ops):
    regs = set()
    for a, b in _VRANGE.findall(ops):
        regs.update(range(int(a), int(b) + 1))
    for r in _VONE.findall(_VRANGE.sub(" ", ops)):
        regs.add(int(r))
    return regs


_LGKM = re.compile(r"lgkmcnt\((\d+)\)")


def untracked_load_violations(insts, load="ds_read_b64_tr_b16"):
    """For every `load`, the instructions reachable from it before a wait
    that covers it and that read or write one of its destination registers.
    A wave's LDS operations complete in issue order, so s_waitcnt
    lgkmcnt(N) covers the load once at least N LDS operations (ds_*) were
    issued after it on the path; other counted operations (scalar loads)
    complete out of order and are not counted."""
    index = {a: i for i, (a, _, _, _) in enumerate(insts)}
    bad = []
    for i, (addr, mnem, ops, _) in enumerate(insts):
        if mnem != load:
            continue
        dest = vregs(ops.split(",")[0])
        seen, stack = set(), [(i + 1, 0)]
        while stack:
            j, later = stack.pop()
            if (j, later) in seen or j >= len(insts):
                continue
            seen.add((j, later))
            a, m, o, tgt = insts[j]
            w = _LGKM.search(o) if m == "s_waitcnt" else None
            if w and later >= int(w.group(1)):
                continue
            if m == load and vregs(o.split(",")[0]) == dest and not (vregs(o.split(",", 1)[1]) & dest):
                # another load into the same registers: the LDS returns one
                # wave's loads in order, so the later value wins (dead reads
                # past the last k-step are allocated this way); keep going
                pass
            elif vregs(o) & dest:
                bad.append((hex(addr), f"{m} {o}"))
                continue
            if m == "s_endpgm":
                continue
            nl = min(later + 1, 16) if m.startswith("ds_") else later
            if tgt is not None:
                stack.append((index[tgt], nl))
            if m != "s_branch":
                stack.append((j + 1, nl))
    return bad


@pytest.fixture(scope="module")
def dumped(tmp_path_factory):
    """Generated sources and code objects of the built-in configurations."""
    if not os.path.exists(OBJDUMP):
        pytest.skip("no ROCm disassembler")
    d = tmp_path_factory.mktemp("lego_dump")
    env = dict(os.environ, LEGO_DUMP=str(d), LEGO_CACHE_DIR=str(d / "cache"), PYTHONPATH=ROOT)
    code = "import paper_2505_08091_amd as L\nprint(L.selftest_compile()[0])\n"
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=900)
    assert r.returncode == 0, r.stderr[-2000:]
    return d


def test_checker_finds_a_planted_early_use():
    """The checker itself: a copy of a destination register before the wait is
    found on the fall-through path and through a loop back-edge; a use after
    the wait is not."""
    text = "\n".join([
        "0000000000001000 <k>:",
        "\tds_read_b64_tr_b16 v[10:11], v3  // 000000001000: 0",
        "\tv_mov_b32_e32 v20, v11  // 000000001008: 0",
        "\ts_waitcnt lgkmcnt(0)  // 00000000100C: 0",
        "\ts_endpgm  // 000000001010: 0",
    ])
    assert len(untracked_load_violations(parse(text))) == 1
    loop = "\n".join([
        "0000000000001000 <k>:",
        "\tv_mov_b32_e32 v20, v11  // 000000001000: 0",
        "\ts_waitcnt lgkmcnt(0)  // 000000001004: 0",
        "\tds_read_b64_tr_b16 v[10:11], v3  // 000000001008: 0",
        "\ts_cbranch_scc0 1  // 000000001010: 0 <k+0x0>",
        "\ts_waitcnt lgkmcnt(0)  // 000000001014: 0",
        "\tv_mov_b32_e32 v21, v10  // 000000001018: 0",
        "\ts_endpgm  // 00000000101C: 0",
    ])
    assert len(untracked_load_violations(parse(loop))) == 1
    ok = loop.replace("\tv_mov_b32_e32 v20, v11  // 000000001000: 0", "\ts_nop 0  // 000000001000: 0")
    assert untracked_load_violations(parse(ok)) == []


def test_checker_counts_later_lds_operations():
    """s_waitcnt lgkmcnt(N) covers a load only when N LDS operations were
    issued after it; a scalar load in between does not count."""
    def prog(between, n):
        lines = ["0000000000001000 <k>:", "\tds_read_b64_tr_b16 v[10:11], v3  // 000000001000: 0"]
        for i, b in enumerate(between):
            lines.append(f"\t{b}  // {0x1008 + 8 * i:012X}: 0")
        lines += [f"\ts_waitcnt lgkmcnt({n})  // 000000001100: 0", "\tv_mov_b32_e32 v20, v11  // 000000001104: 0",
                  "\ts_endpgm  // 000000001108: 0"]
        return parse("\n".join(lines))
    two = ["ds_read_b128 v[20:23], v4", "ds_read2_b32 v[24:25], v5 offset1:2"]
    assert untracked_load_violations(prog(two, 2)) == []
    assert untracked_load_violations(prog(two, 1)) == []
    assert len(untracked_load_violations(prog(two, 3))) == 1
    assert len(untracked_load_violations(prog(two[:1] + ["s_load_dword s4, s[0:1], 0x0"], 2))) == 1


def test_generated_kernels_do_not_spill(dumped):
    """No generated kernel of the built-in configurations spills registers to
    scratch memory (a spill store of a transposing read's destination would
    also read it before its wait)."""
    readelf = os.path.join(os.path.dirname(OBJDUMP), "llvm-readelf")
    n = 0
    for co in sorted(dumped.glob("*.co")):
        notes = subprocess.run([readelf, "--notes", str(co)], capture_output=True, text=True, check=True).stdout
        spills = [int(x) for x in re.findall(r"\.vgpr_spill_count:\s+(\d+)", notes)]
        spills += [int(x) for x in re.findall(r"\.sgpr_spill_count:\s+(\d+)", notes)]
        assert spills and not any(spills), (co.name, spills)
        n += 1
    assert n >= 10


def test_transposing_fragment_reads_are_waited_for(dumped):
    n = 0
    for hip in sorted(dumped.glob("*.hip")):
        src = hip.read_text()
        if "#define A_FRTR 1" not in src and "#define B_FRTR 1" not in src:
            continue
        co = hip.with_suffix(".co")
        text = subprocess.run([OBJDUMP, "-d", "--mcpu=gfx950", str(co)], capture_output=True, text=True,
                              check=True).stdout
        insts = parse(text)
        assert any(m == "ds_read_b64_tr_b16" for _, m, _, _ in insts), hip.name
        bad = untracked_load_violations(insts)
        assert not bad, (hip.name, bad[:5])
        n += 1
    assert n >= 2  # the built-in configurations with m- and n-contiguous operands


HIPCC = "/opt/rocm/bin/hipcc"
BUNDLER = "/opt/rocm/llvm/bin/clang-offload-bundler"


def _gemm_case_ids():
    from tests.test_generated_host import N_GEMM_CASES
    return range(N_GEMM_CASES + len(_measured_gemms(None)))


def _measured_gemms(L):
    """The measured GEMMs that the GPU tests do not launch at these sizes."""
    if L is None:
        return [None] * 6
    n = 8192
    out = [dict(M=8000, N=8000, K=8000, dtype="bf16")]
    for la in ("Row", "Col"):
        for lb in ("Row", "Col"):
            out.append(dict(M=n, N=n, K=n, dtype="f16", a=L.as_layout(getattr(L, la)(n, n)),
                            b=L.as_layout(getattr(L, lb)(n, n))))
    out.append(dict(M=1024, N=1024, K=1024, dtype="f16", bm=128, bn=128, bk=32, wm=64, wn=64))
    return out


@pytest.mark.parametrize("i", _gemm_case_ids())
def test_gemm_configurations_compile_clean(i, tmp_path):
    """Every GEMM configuration the GPU tests launch, and the measured ones,
    compiled for gfx950 with the library's compiler options: no register
    spills, and no transposing read's destination touched before its wait."""
    if not (os.path.exists(HIPCC) and os.path.exists(BUNDLER) and os.path.exists(OBJDUMP)):
        pytest.skip("no ROCm compiler")
    import paper_2505_08091_amd as L
    from tests.test_generated_host import _gemm_cases
    cases = _gemm_cases() + _measured_gemms(L)
    kw = dict(cases[i])
    src = L.plan_source("gemm", **kw)
    hip, co, elf = tmp_path / "k.hip", tmp_path / "k.co", tmp_path / "k.elf"
    hip.write_text(src)
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "--genco", "-Xclang", "-target-feature",
                        "-Xclang", "-packed-fp32-ops", "-include", "hip/hip_runtime.h", str(hip), "-o", str(co)],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    subprocess.run([BUNDLER, "--unbundle", "--type=o", "--targets=hipv4-amdgcn-amd-amdhsa--gfx950",
                    f"--input={co}", f"--output={elf}"], check=True, capture_output=True)
    readelf = os.path.join(os.path.dirname(OBJDUMP), "llvm-readelf")
    notes = subprocess.run([readelf, "--notes", str(elf)], capture_output=True, text=True, check=True).stdout
    spills = [int(x) for x in re.findall(r"\.[vs]gpr_spill_count:\s+(\d+)", notes)]
    assert spills and not any(spills), (kw, spills)
    if "#define A_FRTR 1" in src or "#define B_FRTR 1" in src:
        text = subprocess.run([OBJDUMP, "-d", "--mcpu=gfx950", str(elf)], capture_output=True, text=True,
                              check=True).stdout
        bad = untracked_load_violations(parse(text))
        assert not bad, (kw, bad[:5])
