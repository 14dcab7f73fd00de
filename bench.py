#!/usr/bin/env python3
"""Benchmark of layout-mapped data movement on one MI355X.

Headline workload (one step = one pass of the hot path over one batch): an
8192 x 8192 fp32 tensor (uniform[-1,1), seed 3) remapped from row-major into a
2-level blocked layout (64x64 tiles, column-major tile order, row-major inside
a tile) and back, i.e. two remap launches moving 2 x 512 MiB each.  The value
is whole-job throughput in GB/s (bytes read + bytes written per second) with
the data resident in HBM.

Also reported in the same JSON line:
  gemm          the 8192^3 bf16 tiled GEMM (256x256x64 tiles, grouped + XCD
                schedule, XOR-swizzled LDS) in TFLOP/s with its own roofline;
  roofline      the remap kernel's algorithmic bytes per launch divided by its
                average launch duration (fence-free HIP events between the
                launches of the timed region, on the stream the kernels run on)
                against the 8 TB/s HBM peak;
  cpu_baseline  the CPU oracle timed on this host on a bounded sample;
  more          the other measured workloads (transposing and Morton remaps,
                Morton-A GEMM, the four Row/Col operand layouts of the GEMM).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "layout-remap GB/s (% HBM peak); tiled-GEMM TFLOP/s (% MFMA peak)"
HBM_PEAK_GBPS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
N_REMAP = 8192
N_GEMM = 8192


class HipEvents:
    """Timing events recorded on one HIP stream.

    Created with hipEventDisableSystemFence: a timing-only event then skips the
    system-scope cache write-back and invalidate that an ordinary event performs
    when it completes, which would otherwise stretch the launch after it.  One
    event sits between consecutive launches, so launch j of a sequence lasts
    from event j to event j+1 and the durations add up to the whole region."""
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, n, stream):
        import ctypes
        # The HIP runtime that torch already loaded (no second copy).
        self._hip = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD)
        self._c = ctypes
        self._stream = ctypes.c_void_p(stream)
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            rc = self._hip.hipEventCreateWithFlags(ctypes.byref(e), ctypes.c_uint(self.DISABLE_SYSTEM_FENCE))
            if rc != 0:
                raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")
            self.ev.append(e)

    def record(self, i):
        rc = self._hip.hipEventRecord(self.ev[i], self._stream)
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def ms(self, i, j):
        out = self._c.c_float()
        rc = self._hip.hipEventElapsedTime(self._c.byref(out), self.ev[i], self.ev[j])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return out.value

    def close(self):
        for e in self.ev:
            self._hip.hipEventDestroy(e)
        self.ev = []


def _median(xs):
    xs = sorted(xs)
    m = len(xs) // 2
    return xs[m] if len(xs) % 2 else 0.5 * (xs[m - 1] + xs[m])


def _stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def _source_sha1(L, kind, *args, **kw):
    import hashlib
    return hashlib.sha1(L.plan_source(kind, *args, **kw).encode()).hexdigest()


def profiled_traffic(name, sha1):
    """HBM traffic per launch measured with rocprofv3 (FETCH_SIZE + WRITE_SIZE,
    scaled by the same counters for a copy of known size), read from the
    committed profile summary - only if it was taken on this exact generated
    kernel source; otherwise None."""
    path = os.path.join(ROOT, "profiles", f"{name}.md")
    try:
        with open(path) as f:
            for line in f:
                if line.startswith("traffic-json:"):
                    d = json.loads(line.split(":", 1)[1])
                    if d.get("source_sha1") == sha1:
                        return d["bytes_per_launch"]
    except OSError:
        pass
    return None


def bench_remap(L, steps, warmup):
    import torch
    import synth_inputs as S
    n = N_REMAP
    src = S.tensor(n * n, "f32", seed=S.SEED_SRC).cuda()
    blk_buf = torch.empty_like(src)
    back = torch.empty_like(src)
    row = L.as_layout(L.Row(n, n))
    blk = L.TileOrderBy(L.Col(n // 64, n // 64), L.Row(64, 64))
    plan_f = L.remap_plan(row, blk, 4)
    plan_b = L.remap_plan(blk, row, 4)
    for _ in range(warmup):
        L.remap(row, blk, src, blk_buf)
        L.remap(blk, row, blk_buf, back)
    # Timed region: `steps` x (forward, inverse), one event between launches.
    ev = HipEvents(2 * steps + 1, _stream())
    torch.cuda.synchronize()
    for k in range(steps):
        ev.record(2 * k)
        L.remap(row, blk, src, blk_buf)
        ev.record(2 * k + 1)
        L.remap(blk, row, blk_buf, back)
    ev.record(2 * steps)
    torch.cuda.synchronize()
    total_ms = ev.ms(0, 2 * steps)
    fwd = [ev.ms(2 * k, 2 * k + 1) for k in range(steps)]
    inv = [ev.ms(2 * k + 1, 2 * k + 2) for k in range(steps)]
    ev.close()
    assert torch.equal(back, src), "remap round trip is not the identity"
    # Practical copy ceiling: the identity remap (a plain vector copy) of the
    # same bytes, alternating directions like the timed region.
    for _ in range(10):
        L.remap(row, row, src, back)
        L.remap(row, row, back, blk_buf)
    cev = HipEvents(41, _stream())
    torch.cuda.synchronize()
    for k in range(20):
        cev.record(2 * k)
        L.remap(row, row, src, back)
        cev.record(2 * k + 1)
        L.remap(row, row, back, blk_buf)
    cev.record(40)
    torch.cuda.synchronize()
    copy_ms = cev.ms(0, 40) / 40
    cev.close()
    return {
        "sha1": _source_sha1(L, "remap", row, blk, param=4),
        "total_ms": total_ms,
        "launch_ms": (sum(fwd) + sum(inv)) / (2 * steps),
        "launch_median_ms": _median(fwd + inv),
        "launch_min_ms": min(fwd + inv),
        "fwd_ms": sum(fwd) / steps,
        "inv_ms": sum(inv) / steps,
        "copy_ms": copy_ms,
        "bytes_per_launch": 2 * n * n * 4,
        "plan_fwd": plan_f["info"],
        "plan_inv": plan_b["info"],
    }


def bench_gemm(L, steps, warmup):
    import torch
    import synth_inputs as S
    n = N_GEMM
    a = S.tensor(n * n, "bf16", dist="normal", seed=S.SEED_A).cuda()
    b = S.tensor(n * n, "bf16", dist="normal", seed=S.SEED_B).cuda()
    c = torch.empty(n * n, dtype=torch.float32, device="cuda")
    # Operand and MFMA fragment layouts given explicitly as layouts (A row-major,
    # B column-major, C row-major, the 32x32x16 fragments); the schedule and the
    # LDS layouts are the planner's grouped + XCD order and XOR swizzles.
    kw = dict(a=L.as_layout(L.Row(n, n)), b=L.as_layout(L.Col(n, n)), c=L.as_layout(L.Row(n, n)),
              frag_a=L.mfma_fragment_layout(0, 0), frag_b=L.mfma_fragment_layout(0, 1),
              frag_c=L.mfma_fragment_layout(0, 2))
    plan = L.gemm_plan(n, n, n, "bf16", **kw)
    for _ in range(warmup):
        L.gemm(a, b, c, n, n, n, "bf16", **kw)
    ev = HipEvents(steps + 1, _stream())
    torch.cuda.synchronize()
    for k in range(steps):
        ev.record(k)
        L.gemm(a, b, c, n, n, n, "bf16", **kw)
    ev.record(steps)
    torch.cuda.synchronize()
    ms = ev.ms(0, steps) / steps
    each = [ev.ms(k, k + 1) for k in range(steps)]
    ev.close()
    flops = 2.0 * n ** 3
    tf = flops / (ms * 1e-3) / 1e12
    return {"ms": ms, "median_ms": _median(each), "min_ms": min(each), "tflops": tf, "plan": plan, "a": a, "b": b, "c": c,
            "sha1": _source_sha1(L, "gemm", M=n, N=n, K=n, dtype="bf16", **kw)}


def _alternate(L, la, lb, x, y, z, reps, warmup=5):
    """Remaps la->lb (x -> y) and lb->la (y -> z), alternating, one event
    between launches; mean ms of each direction.  z must equal x."""
    import torch
    for _ in range(warmup):
        L.remap(la, lb, x, y)
        L.remap(lb, la, y, z)
    ev = HipEvents(2 * reps + 1, _stream())
    torch.cuda.synchronize()
    for k in range(reps):
        ev.record(2 * k)
        L.remap(la, lb, x, y)
        ev.record(2 * k + 1)
        L.remap(lb, la, y, z)
    ev.record(2 * reps)
    torch.cuda.synchronize()
    f = sum(ev.ms(2 * k, 2 * k + 1) for k in range(reps)) / reps
    i = sum(ev.ms(2 * k + 1, 2 * k + 2) for k in range(reps)) / reps
    ev.close()
    assert torch.equal(z, x), "remap round trip is not the identity"
    return f, i


def _alone(L, la, lb, x, y, reps, warmup=5):
    """Mean ms of the remap la->lb (x -> y) launched `reps` times in a row."""
    import torch
    for _ in range(warmup):
        L.remap(la, lb, x, y)
    ev = HipEvents(reps + 1, _stream())
    torch.cuda.synchronize()
    for k in range(reps):
        ev.record(k)
        L.remap(la, lb, x, y)
    ev.record(reps)
    torch.cuda.synchronize()
    ms = ev.ms(0, reps) / reps
    ev.close()
    return ms


def _flushed(L, la, lb, x, y, z, scratch, reps):
    """Like _alternate, but a 1 GiB fill (not timed) evicts the 256 MB
    last-level cache before every launch."""
    import torch
    ev = HipEvents(4 * reps, _stream())
    torch.cuda.synchronize()
    for k in range(reps):
        scratch.fill_(k)
        ev.record(4 * k)
        L.remap(la, lb, x, y)
        ev.record(4 * k + 1)
        scratch.fill_(k + 0.5)
        ev.record(4 * k + 2)
        L.remap(lb, la, y, z)
        ev.record(4 * k + 3)
    torch.cuda.synchronize()
    f = sum(ev.ms(4 * k, 4 * k + 1) for k in range(reps)) / reps
    i = sum(ev.ms(4 * k + 2, 4 * k + 3) for k in range(reps)) / reps
    ev.close()
    assert torch.equal(z, x), "remap round trip is not the identity"
    return f, i


def _gemm_ms(L, a_buf, b_buf, c_buf, n, dtype, reps, warmup=30, **kw):
    """Mean launch duration after ``warmup`` untimed launches (the shader
    clock needs ~20 back-to-back large GEMMs to settle)."""
    import torch
    for _ in range(warmup):
        L.gemm(a_buf, b_buf, c_buf, n, n, n, dtype, **kw)
    ev = HipEvents(reps + 1, _stream())
    torch.cuda.synchronize()
    for k in range(reps):
        ev.record(k)
        L.gemm(a_buf, b_buf, c_buf, n, n, n, dtype, **kw)
    ev.record(reps)
    torch.cuda.synchronize()
    ms = ev.ms(0, reps) / reps
    ev.close()
    return ms


def bench_extra(L, reps=20):
    """The other measured workloads: index maps of the blocked layout on the
    device, the 128^3 and 1024^3 GEMMs, transposing remaps (Row <-> Col fp32,
    the 2D transpose of Section V-C), Row <-> Morton fp16 4096^2 hot and with
    the last-level cache flushed, the 4096^3 fp16 GEMM with A in Morton order
    and B row-major, the four Row/Col operand layouts of an 8192^3 fp16 GEMM
    (Section V-A), workgroup schedules given as layouts (grouped, row-major,
    Morton; Section II), partial tiles: a padding/cropping remap and an 8000^3
    GEMM (Section III-D), 3-D bricks of a 512^3 grid, and user-defined GenPs from expression text: a
    wavefront tile order and an LDS swizzle (Section III-B)."""
    import torch
    import synth_inputs as S

    def gbps(nbytes, ms):
        return round(nbytes / (ms * 1e-3) / 1e9, 1)

    out = {}
    # Index maps on the device (out[x] = apply(x), out[p] = inv(p)) of the
    # 8192^2 blocked layout, int32 outputs: pure write streams.
    n = 8192
    blk = L.TileOrderBy(L.Col(n // 64, n // 64), L.Row(64, 64))
    o1 = torch.empty(n * n, dtype=torch.int32, device="cuda")
    o2 = torch.empty(2 * n * n, dtype=torch.int32, device="cuda")
    for _ in range(5):
        L.apply_all_device(blk, o1)
        L.inv_all_device(blk, o2)
    ev = HipEvents(2 * reps + 1, _stream())
    torch.cuda.synchronize()
    for k in range(reps):
        ev.record(2 * k)
        L.apply_all_device(blk, o1)
        ev.record(2 * k + 1)
        L.inv_all_device(blk, o2)
    ev.record(2 * reps)
    torch.cuda.synchronize()
    fa = sum(ev.ms(2 * k, 2 * k + 1) for k in range(reps)) / reps
    fi = sum(ev.ms(2 * k + 1, 2 * k + 2) for k in range(reps)) / reps
    ev.close()
    out["index_maps_i32_8192_blocked"] = {"apply_bytes": 4 * n * n, "apply_GBps": gbps(4 * n * n, fa),
                                          "inv_bytes": 8 * n * n, "inv_GBps": gbps(8 * n * n, fi),
                                          "frac_hbm": round((12 * n * n) / ((fa + fi) * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)}
    del o1, o2

    # The smaller GEMM configurations: 128^3 fp16 with 64x64 tiles of 16x16
    # wave tiles, and 1024^3 fp16 with 128x128x32 tiles, 64x64 wave tiles and
    # a group of 8 (launch-bound: 64 workgroups on 256 CUs).
    small = {}
    for n, kw in ((128, dict(bm=64, bn=64, bk=32, wm=16, wn=16)),
                  (1024, dict(bm=128, bn=128, bk=32, wm=64, wn=64, group_m=8))):
        a = S.tensor(n * n, "f16", seed=S.SEED_A).cuda()
        b = S.tensor(n * n, "f16", seed=S.SEED_B).cuda()
        c = torch.empty(n * n, dtype=torch.float32, device="cuda")
        ms = _gemm_ms(L, a, b, c, n, "f16", reps, **kw)
        small[f"f16_{n}"] = {"us": round(ms * 1e3, 2), "tflops": round(2.0 * n ** 3 / (ms * 1e-3) / 1e12, 2),
                             "plan": L.gemm_plan(n, n, n, "f16", **kw)}
    out["gemm_small"] = small

    tr = []
    for n in (2048, 4096, 8192):
        x = S.tensor(n * n, "f32", seed=S.SEED_SRC).cuda()
        y, z = torch.empty_like(x), torch.empty_like(x)
        row, col = L.as_layout(L.Row(n, n)), L.as_layout(L.Col(n, n))
        # the two directions alternating (each reads the other's output, as
        # a round trip does), and each launched repeatedly on its own source:
        # the caches treat the two patterns differently (at 2048^2 the row ->
        # column kernel that follows a column -> row launch runs twice as
        # long, equal bytes; at 8192^2 a repeated source stays partly in the
        # 256 MB last-level cache)
        f, i = _alternate(L, row, col, x, y, z, reps)
        fa = _alone(L, row, col, x, y, reps)
        ia = _alone(L, col, row, y, z, reps)
        nb = 2 * n * n * 4
        tr.append({"n": n, "bytes_per_launch": nb, "row_to_col_GBps": gbps(nb, f), "col_to_row_GBps": gbps(nb, i),
                   "frac_hbm": round(2 * nb / ((f + i) * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                   "alone_row_to_col_GBps": gbps(nb, fa), "alone_col_to_row_GBps": gbps(nb, ia),
                   "plan": L.remap_plan(row, col, 4)["info"]})
        del x, y, z
    out["transpose_f32"] = tr

    n = 4096
    x = S.tensor(n * n, "f16", seed=S.SEED_SRC).cuda()
    y, z = torch.empty_like(x), torch.empty_like(x)
    row, mz = L.as_layout(L.Row(n, n)), L.as_layout(L.GenP("morton", [n, n]))
    nb = 2 * n * n * 2
    f, i = _alternate(L, row, mz, x, y, z, reps)
    scratch = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    ff, fi = _flushed(L, row, mz, x, y, z, scratch, reps)
    # The practical ceiling at this size: the identity remap (a plain vector
    # copy of the same 64 MiB per launch), hot and flushed.
    cf, ci = _alternate(L, row, row, x, y, z, reps)
    cff, cfi = _flushed(L, row, row, x, y, z, scratch, reps)
    del scratch
    out["morton_f16_4096"] = {"bytes_per_launch": nb, "hot_row_to_morton_GBps": gbps(nb, f),
                              "hot_morton_to_row_GBps": gbps(nb, i), "flushed_row_to_morton_GBps": gbps(nb, ff),
                              "flushed_morton_to_row_GBps": gbps(nb, fi),
                              "identity_copy_hot_GBps": gbps(nb, (cf + ci) / 2),
                              "identity_copy_flushed_GBps": gbps(nb, (cff + cfi) / 2),
                              "plan": L.remap_plan(row, mz, 2)["info"]}

    a_log = S.tensor(n * n, "f16", seed=S.SEED_A).cuda()
    a_mz = torch.empty_like(a_log)
    L.remap(row, mz, a_log, a_mz)
    b = S.tensor(n * n, "f16", seed=S.SEED_B).cuda()
    c = torch.empty(n * n, dtype=torch.float32, device="cuda")
    kw = dict(a=mz, b=L.as_layout(L.Row(n, n)))
    ms = _gemm_ms(L, a_mz, b, c, n, "f16", reps, **kw)
    tf = 2.0 * n ** 3 / (ms * 1e-3) / 1e12
    out["gemm_morton_a_f16_4096"] = {"tflops": round(tf, 1), "frac_mfma": round(tf / BF16_PEAK_TFLOPS, 4),
                                     "plan": L.gemm_plan(n, n, n, "f16", **kw)}
    del a_log, a_mz, b, c

    n = 8192
    a = S.tensor(n * n, "f16", seed=S.SEED_A).cuda()
    b = S.tensor(n * n, "f16", seed=S.SEED_B).cuda()
    c = torch.empty(n * n, dtype=torch.float32, device="cuda")
    var = {}
    for la in ("Row", "Col"):
        for lb in ("Row", "Col"):
            kw = dict(a=L.as_layout(getattr(L, la)(n, n)), b=L.as_layout(getattr(L, lb)(n, n)))
            ms = _gemm_ms(L, a, b, c, n, "f16", 20, **kw)
            var[f"A {la} B {lb}"] = round(2.0 * n ** 3 / (ms * 1e-3) / 1e12, 1)
    out["gemm_operand_layouts_f16_8192_tflops"] = var
    del a, b, c

    # Workgroup schedules given as layouts over the 32 x 32 tile grid of the
    # 8192^3 bf16 GEMM (Section II: the grouped order against row-major).
    a = S.tensor(n * n, "bf16", dist="normal", seed=S.SEED_A).cuda()
    b = S.tensor(n * n, "bf16", dist="normal", seed=S.SEED_B).cuda()
    c = torch.empty(n * n, dtype=torch.float32, device="cuda")
    t = n // 256
    sch = {}
    for name, kw in (("grouped 8 + XCD remap (default)", {}),
                     ("grouped 8", dict(xcd_remap=0)),
                     ("row-major", dict(sched=L.as_layout(L.Row(t, t)), xcd_remap=0)),
                     ("row-major + XCD remap", dict(sched=L.as_layout(L.Row(t, t)))),
                     ("Morton", dict(sched=L.as_layout(L.GenP("morton", [t, t])), xcd_remap=0))):
        ms = _gemm_ms(L, a, b, c, n, "bf16", 20, **kw)
        sch[name] = round(2.0 * n ** 3 / (ms * 1e-3) / 1e12, 1)
    out["gemm_schedules_bf16_8192_tflops"] = sch
    del a, b, c

    # Partial tiles (ExpandBy, Section III-D): an 8000 x 8000 fp32 array into a
    # zero-padded 8192 x 8192 blocked buffer and back, and an 8000^3 bf16 GEMM
    # whose 256-wide tiles overhang the matrices.
    n, ne = 8000, 8192
    x = S.tensor(n * n, "f32", seed=S.SEED_SRC).cuda()
    padded = torch.empty(ne * ne, dtype=torch.float32, device="cuda")
    z = torch.empty_like(x)
    src = L.ExpandBy([n, n], [ne, ne], L.as_layout(L.Row(ne, ne)))
    blk = L.TileOrderBy(L.Col(ne // 64, ne // 64), L.Row(64, 64))
    f, i = _alternate(L, src, blk, x, padded, z, reps)
    # bytes the kernels must move: pad reads n^2 and writes ne^2; crop the reverse
    nb = (n * n + ne * ne) * 4
    out["pad_crop_f32_8000_in_8192"] = {"bytes_per_launch": nb, "pad_GBps": gbps(nb, f), "crop_GBps": gbps(nb, i),
                                        "frac_hbm": round(2 * nb / ((f + i) * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                                        "plan_pad": L.remap_plan(src, blk, 4)["info"],
                                        "plan_crop": L.remap_plan(blk, src, 4)["info"]}
    del x, padded, z
    a = S.tensor(n * n, "bf16", dist="normal", seed=S.SEED_A).cuda()
    b = S.tensor(n * n, "bf16", dist="normal", seed=S.SEED_B).cuda()
    c = torch.empty(n * n, dtype=torch.float32, device="cuda")
    ms = _gemm_ms(L, a, b, c, n, "bf16", 20)
    tf = 2.0 * n ** 3 / (ms * 1e-3) / 1e12
    out["gemm_ragged_bf16_8000"] = {"tflops": round(tf, 1), "frac_mfma": round(tf / BF16_PEAK_TFLOPS, 4),
                                    "plan": L.gemm_plan(n, n, n, "bf16")}
    del a, b, c

    # A whole matrix in antidiagonal order (Figure 7's GenP, the wavefront
    # order of Section V's NW example) and back: no digit structure, so the
    # box path (square boxes of the index space through LDS).
    for n, dt in ((4096, "f32"), (8192, "f32"), (4096, "f16")):
        x = S.tensor(n * n, dt, seed=S.SEED_SRC).cuda()
        y, z = torch.empty_like(x), torch.empty_like(x)
        row, ad = L.as_layout(L.Row(n, n)), L.as_layout(L.GenP("antidiag", [n, n]))
        f, i = _alternate(L, row, ad, x, y, z, reps)
        nb = 2 * n * n * x.element_size()
        out[f"antidiagonal_{dt}_{n}"] = {"bytes_per_launch": nb, "row_to_antidiag_GBps": gbps(nb, f),
                                         "antidiag_to_row_GBps": gbps(nb, i),
                                         "frac_hbm": round(2 * nb / ((f + i) * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                                         "plan": L.remap_plan(row, ad, x.element_size())["info"]}
        del x, y, z

    # 3-D bricks (the stencil data layout of Section V): a 512^3 fp32 grid
    # between row-major order and bricks of 8^3 or 4^3 elements stored
    # contiguously, bricks in row-major order.
    n = 512
    x = S.tensor(n ** 3, "f32", seed=S.SEED_SRC).cuda()
    y, z = torch.empty_like(x), torch.empty_like(x)
    row = L.as_layout(L.Row(n, n, n))
    br = []
    for b in (8, 4):
        bricks = L.TileOrderBy(L.Row(n // b, n // b, n // b), L.Row(b, b, b))
        f, i = _alternate(L, row, bricks, x, y, z, reps)
        nb = 2 * n ** 3 * 4
        br.append({"brick": b, "bytes_per_launch": nb, "row_to_bricks_GBps": gbps(nb, f),
                   "bricks_to_row_GBps": gbps(nb, i),
                   "frac_hbm": round(2 * nb / ((f + i) * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                   "plan": L.remap_plan(row, bricks, 4)["info"]})
    out["bricks_f32_512cubed"] = br
    del x, y, z

    # User-defined GenPs from expression text: an 8192^2 fp32 array whose 64x64
    # tiles are stored in antidiagonal (wavefront) order, and the 8192^3 bf16
    # GEMM with its LDS swizzle written as an expression.
    n, t = 8192, 64
    q = n // t
    antidiag = ("i + j < n0 ? i + (i + j) * (i + j + 1) / 2 : n0 * n0 - 1 - ((n0 - 1 - i) + "
                "(2 * n0 - 2 - i - j) * (2 * n0 - 1 - i - j) / 2)")
    tri = "(isqrt(8 * {y} + 1) - 1) / 2"
    row_of = "({y} - " + tri + " * (" + tri + " + 1) / 2)"
    up, y2 = "x < n0 * (n0 + 1) / 2", "(n0 * n0 - 1 - x)"
    inv = [f"{up} ? {row_of.format(y='x')} : n0 - 1 - {row_of.format(y=y2)}",
           f"{up} ? ({tri.format(y='x')} - {row_of.format(y='x')}) : "
           f"n0 - 1 - ({tri.format(y=y2)} - {row_of.format(y=y2)})"]
    wave = L.GroupBy([n, n]).OrderBy(L.RegP([q, t, q, t], [1, 3, 2, 4])).OrderBy(
        L.GenPExpr([q, q], antidiag, inv), L.Row(t, t))
    row = L.as_layout(L.Row(n, n))
    x = S.tensor(n * n, "f32", seed=S.SEED_SRC).cuda()
    y, z = torch.empty_like(x), torch.empty_like(x)
    f, i = _alternate(L, row, wave, x, y, z, reps)
    nb = 2 * n * n * 4
    out["wavefront_tiles_f32_8192"] = {"bytes_per_launch": nb, "row_to_wavefront_GBps": gbps(nb, f),
                                       "wavefront_to_row_GBps": gbps(nb, i),
                                       "frac_hbm": round(2 * nb / ((f + i) * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                                       "plan": L.remap_plan(row, wave, 4)["info"]}
    del x, y, z
    a = S.tensor(n * n, "bf16", dist="normal", seed=S.SEED_A).cuda()
    b = S.tensor(n * n, "bf16", dist="normal", seed=S.SEED_B).cuda()
    c = torch.empty(n * n, dtype=torch.float32, device="cuda")
    sw = L.as_layout(L.GenPExpr([256, 64], "i * 64 + (((j / 8) ^ ((i / 2) % 8)) * 8) + j % 8",
                                ["x / 64", "(((x % 64) / 8) ^ ((x / 128) % 8)) * 8 + x % 8"]))
    ms = _gemm_ms(L, a, b, c, n, "bf16", 20, lds_a=sw, lds_b=sw)
    tf = 2.0 * n ** 3 / (ms * 1e-3) / 1e12
    out["gemm_expression_lds_bf16_8192"] = {"tflops": round(tf, 1), "frac_mfma": round(tf / BF16_PEAK_TFLOPS, 4),
                                            "plan": L.gemm_plan(n, n, n, "bf16", lds_a=sw, lds_b=sw)}
    return out


def _remap_pair(L, name):
    """The two layouts, element size and size of a named remap workload."""
    kind, dt, n = name.split("_")[0], name.split("_")[1], int(name.split("_")[2])
    row = L.as_layout(L.Row(n, n))
    other = {"transpose": lambda: L.as_layout(L.Col(n, n)),
             "morton": lambda: L.as_layout(L.GenP("morton", [n, n])),
             "antidiag": lambda: L.as_layout(L.GenP("antidiag", [n, n])),
             "blocked": lambda: L.TileOrderBy(L.Col(n // 64, n // 64), L.Row(64, 64)),
             "identity": lambda: row}[kind]()
    return row, other, dt, n


WORKLOADS = ("remap: blocked_f32_8192, transpose_f32_{2048,4096,8192}, morton_f16_4096, antidiag_f32_{4096,8192}, "
             "identity_f32_8192 (a plain copy) "
             "(suffix _fwd or _inv: one direction only, its source fixed; _flushed: a 1 GiB fill evicts the "
             "last-level cache before each launch); gemm: gemm_bf16_8192 (the measured GEMM), "
             "gemm_<f16|bf16>_<n>_<A>_<B> with A, B each row, col or morton")


def run_workload(L, name, reps):
    """``reps`` launches of one named workload and nothing else (for
    rocprofv3 runs; see WORKLOADS).  Remaps alternate directions unless a
    direction is named; returns the mean duration of each direction."""
    import torch
    import synth_inputs as S
    if name == "gemm_bf16_8192":
        g = bench_gemm(L, reps, 30)
        return {"workload": name, "ms": round(g["ms"], 5), "tflops": round(g["tflops"], 1), "plan": g["plan"]}
    if name.startswith("gemm_"):
        # gemm_<dtype>_<n>_<A>_<B>, A and B each row, col or morton
        _, dt, n, la, lb = name.split("_")
        n = int(n)
        a = S.tensor(n * n, dt, dist="normal", seed=S.SEED_A).cuda()
        b = S.tensor(n * n, dt, dist="normal", seed=S.SEED_B).cuda()
        c = torch.empty(n * n, dtype=torch.float32, device="cuda")
        lay = {"row": lambda: L.as_layout(L.Row(n, n)), "col": lambda: L.as_layout(L.Col(n, n)),
               "morton": lambda: L.as_layout(L.GenP("morton", [n, n]))}
        kw = dict(a=lay[la](), b=lay[lb]())
        # the operands' values are those of a row-major matrix, stored in each layout
        if la != "row":
            t = torch.empty_like(a)
            L.remap(lay["row"](), kw["a"], a, t)
            a = t
        if lb != "row":
            t = torch.empty_like(b)
            L.remap(lay["row"](), kw["b"], b, t)
            b = t
        ms = _gemm_ms(L, a, b, c, n, dt, reps, warmup=10, **kw)
        return {"workload": name, "ms": round(ms, 5), "tflops": round(2.0 * n ** 3 / ms / 1e9, 1),
                "plan": L.gemm_plan(n, n, n, dt, **kw)}
    base = name.replace("_fwd", "").replace("_inv", "").replace("_flushed", "")
    row, other, dt, n = _remap_pair(L, base)
    x = S.tensor(n * n, dt, seed=S.SEED_SRC).cuda()
    y, z = torch.empty_like(x), torch.empty_like(x)
    nb = 2 * n * n * x.element_size()
    if name.endswith("_fwd") or name.endswith("_inv"):
        la, lb = (row, other) if name.endswith("_fwd") else (other, row)
        if name.endswith("_inv"):
            L.remap(row, other, x, z)
            x, z = z, x
        ms = _alone(L, la, lb, x, y, reps)
        return {"workload": name, "ms": round(ms, 5), "GBps": round(nb / ms / 1e6, 1),
                "plan": L.remap_plan(la, lb, x.element_size())["info"]}
    if name.endswith("_flushed"):
        L.remap(row, other, x, y)  # load both kernels before the timed launches
        L.remap(other, row, y, z)
        scratch = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        f, i = _flushed(L, row, other, x, y, z, scratch, reps)
    else:
        f, i = _alternate(L, row, other, x, y, z, reps)
    return {"workload": name, "fwd_ms": round(f, 5), "inv_ms": round(i, 5), "fwd_GBps": round(nb / f / 1e6, 1),
            "inv_GBps": round(nb / i / 1e6, 1), "plan_fwd": L.remap_plan(row, other, x.element_size())["info"],
            "plan_inv": L.remap_plan(other, row, x.element_size())["info"]}


def cpu_baseline_remap(rounds=2):
    """The oracle remap of the full 8192^2 fp32 tensor, forward and back,
    ``rounds`` times, timed on this host."""
    import synth_inputs as S
    from oracle import layout as OL
    from oracle import remap as OR
    n = N_REMAP
    src = S.tensor(n * n, "f32", seed=S.SEED_SRC).numpy()
    row = OL.as_layout(OL.Row(n, n))
    blk = OL.TileOrderBy(OL.Col(n // 64, n // 64), OL.Row(64, 64))
    t = time.perf_counter()
    for _ in range(rounds):
        back = OR.remap(blk, row, OR.remap(row, blk, src))
    dt = time.perf_counter() - t
    assert (back == src).all()
    moved = rounds * 2 * (2 * n * n * 4)
    return {"value": round(moved / dt / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{rounds} x (forward + inverse) remap of the whole {n}x{n} fp32 tensor, {moved >> 20} MiB "
                      f"moved in {dt:.1f} s; numpy element-wise and gather kernels run on one thread "
                      f"(host has {len(os.sched_getaffinity(0))} cores)"}


def cpu_baseline_gemm(a, b, min_s=10.0, max_reps=5):
    """The oracle fp64 GEMM of the whole 8192^3 problem, repeated until
    ``min_s`` seconds have passed (at most ``max_reps`` times)."""
    import synth_inputs as S
    from oracle import gemm as OG
    from oracle import layout as OL
    n = N_GEMM
    a_np = S.as_numpy_bits(a.cpu())
    b_np = S.as_numpy_bits(b.cpu())
    la, lb = OL.as_layout(OL.Row(n, n)), OL.as_layout(OL.Col(n, n))
    reps = 0
    t = time.perf_counter()
    while reps < max_reps and (reps == 0 or time.perf_counter() - t < min_s):
        OG.gemm(a_np, b_np, la, lb, "bf16")
        reps += 1
    dt = time.perf_counter() - t
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    return {"value": round(reps * 2.0 * n ** 3 / dt / 1e12, 5), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} x the whole bf16 {n}^3 GEMM in fp64 ({dt:.1f} s, operand decode through the "
                      f"layouts included; the fp64 product runs in numpy's BLAS)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--gemm-steps", type=int, default=50)
    # The shader clock settles only after ~20 back-to-back 8192^3 GEMMs (about
    # 20 ms of full MFMA load); earlier launches run ~12% slower.
    ap.add_argument("--gemm-warmup", type=int, default=40)
    ap.add_argument("--no-gemm", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="skip the other workloads (transposes, Morton, "
                                                            "operand-layout GEMMs)")
    ap.add_argument("--workload", help="run only this workload, --steps launches (for profiling): " + WORKLOADS)
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the layout remap and GEMM kernels run on a single MI355X; "
              "multi-GPU sharding is a design note, not a measured path.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2505_08091_amd as L
    torch.cuda.set_device(0)
    if args.workload:
        print(json.dumps(run_workload(L, args.workload, args.steps)), flush=True)
        return

    r = bench_remap(L, args.steps, args.warmup)
    ms_step = r["total_ms"] / args.steps
    value = 2 * r["bytes_per_launch"] / (ms_step * 1e-3) / 1e9
    achieved = r["bytes_per_launch"] / (r["launch_ms"] * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "layout remap of an 8192x8192 fp32 tensor, row-major -> 2-level blocked (64x64 tiles, "
                        "column-major tile order, row-major inside tiles) and back; one step = forward + inverse",
            "elements": N_REMAP * N_REMAP,
            "bytes_per_step": 2 * r["bytes_per_launch"],
            "plan_forward": r["plan_fwd"],
            "plan_inverse": r["plan_inv"],
            "forward_ms": round(r["fwd_ms"], 5),
            "inverse_ms": round(r["inv_ms"], 5),
            "identity_copy_GBps": round(r["bytes_per_launch"] / (r["copy_ms"] * 1e-3) / 1e9, 1),
        },
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": profiled_traffic("remap_direct_8192x8192_f32_row_to_blocked", r["sha1"]),
                     "kernel": "lego_remap_direct", "bytes_per_launch": r["bytes_per_launch"],
                     "avg_launch_ms": round(r["launch_ms"], 5),
                     "median_launch_ms": round(r["launch_median_ms"], 5),
                     "min_launch_ms": round(r["launch_min_ms"], 5)},
    }
    if not args.no_gemm:
        g = bench_gemm(L, args.gemm_steps, args.gemm_warmup)
        out["gemm"] = {
            "metric": "tiled-GEMM TFLOP/s", "value": round(g["tflops"], 1), "unit": "TFLOP/s", "dtype": "bf16",
            "workload": "bf16 GEMM M=N=K=8192, fp32 accumulation and fp32 C, A row-major, B column-major, "
                        "256x256x64 tiles, grouped (8) + XCD schedule, XOR-swizzled LDS, 32x32x16 MFMA fragment layouts given as layouts",
            "plan": g["plan"], "steps": args.gemm_steps, "warmup": args.gemm_warmup,
            "roofline": {"bound": "mfma", "achieved": round(g["tflops"], 1), "peak": BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(g["tflops"] / BF16_PEAK_TFLOPS, 4),
                         "traffic": profiled_traffic("gemm_8192_bf16", g["sha1"]),
                         "kernel": "lego_gemm", "flops_per_launch": 2 * N_GEMM ** 3,
                         "avg_launch_ms": round(g["ms"], 5), "median_launch_ms": round(g["median_ms"], 5),
                         "min_launch_ms": round(g["min_ms"], 5)},
        }
        if not args.no_cpu_baseline:
            out["gemm"]["cpu_baseline"] = cpu_baseline_gemm(g["a"], g["b"])
    if not args.no_extra:
        out["more"] = bench_extra(L)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_remap()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
