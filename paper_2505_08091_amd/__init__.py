"""Python binding of liblego.so (include/lego.h): argument marshalling only.

Every computation happens in the native library and its generated gfx950
kernels.  torch is used only to pass device pointers and the current stream.
Importing this module loads ``liblego.so`` from this directory and raises
ImportError if it has not been built (``python -m paper_2505_08091_amd.build``
or ``__graft_entry__.build()``); there is no fallback.

Layouts follow the paper's notation::

    L = GroupBy([6, 6]).OrderBy(RegP([2, 3, 2, 3], [1, 3, 2, 4])) \
                       .OrderBy(RegP([2, 2], [2, 1]), GenP("antidiag", [3, 3]))
    L.apply([4, 2]) == 15 and L.inv(15) == [4, 2]
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIBPATH = os.path.join(_HERE, "liblego.so")
if not os.path.exists(_LIBPATH):
    raise ImportError(f"{_LIBPATH} is missing: build it with __graft_entry__.build()")
# The library must bind to the HIP runtime that torch loads.  Loaded first,
# it would bring in the system's HIP and HSA runtimes and torch would then
# load its own: two runtimes in one process, and the second one to open the
# GPU finds no device.  torch loaded first provides the runtime's soname,
# which the library's dependency then resolves to.
try:
    import torch  # noqa: F401
except ImportError:
    pass
_lib = ctypes.CDLL(_LIBPATH)

c_i64p = ctypes.POINTER(ctypes.c_int64)
c_i32p = ctypes.POINTER(ctypes.c_int32)
_vp = ctypes.c_void_p

LEGO_OK = 0
STATUS = {0: "OK", -1: "INVALID_ARG", -2: "SIZE_MISMATCH", -3: "NOT_PERMUTATION", -4: "OUT_OF_RANGE",
          -5: "NOT_BIJECTIVE", -6: "UNSUPPORTED", -7: "JIT", -8: "HIP", -9: "NO_MEMORY"}
GENP = {"morton": 1, "xor_swizzle": 2, "reverse": 3, "antidiag": 4}
DTYPES = {"f32": 0, "f16": 1, "bf16": 2}


class LegoError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code
        self.status = STATUS.get(code, str(code))


class lego_gemm_desc(ctypes.Structure):  # noqa: N801 (C name)
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("in_dtype", ctypes.c_int), ("bm", ctypes.c_int), ("bn", ctypes.c_int), ("bk", ctypes.c_int),
                ("wm", ctypes.c_int), ("wn", ctypes.c_int), ("group_m", ctypes.c_int), ("xcd_remap", ctypes.c_int),
                ("stages", ctypes.c_int), ("max_workgroups", ctypes.c_int), ("a", _vp), ("b", _vp), ("c", _vp), ("sched", _vp), ("lds_a", _vp), ("lds_b", _vp),
                ("frag_a", _vp), ("frag_b", _vp), ("frag_c", _vp)]


_SIGS = {
    "lego_last_error": ([], ctypes.c_char_p),
    "lego_version": ([], ctypes.c_char_p),
    "lego_retain": ([_vp], None),
    "lego_release": ([_vp], None),
    "lego_regp": ([ctypes.c_int, c_i64p, c_i32p, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_row": ([ctypes.c_int, c_i64p, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_col": ([ctypes.c_int, c_i64p, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_genp": ([ctypes.c_int, ctypes.c_int, c_i64p, c_i64p, ctypes.c_int, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_genp_expr": ([ctypes.c_int, c_i64p, ctypes.c_char_p, ctypes.c_char_p, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_piece_dims": ([_vp, ctypes.POINTER(ctypes.c_int), c_i64p], ctypes.c_int),
    "lego_groupby": ([ctypes.c_int, c_i64p, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_groupby_tiles": ([ctypes.c_int, ctypes.c_int, c_i64p, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_orderby": ([_vp, ctypes.c_int, ctypes.POINTER(_vp), ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_tileby": ([ctypes.c_int, ctypes.c_int, c_i64p, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_tileorderby": ([ctypes.c_int, ctypes.c_int, ctypes.POINTER(_vp), ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_layout_from_piece": ([_vp, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_expandby": ([ctypes.c_int, c_i64p, c_i64p, _vp, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_layout_rank": ([_vp, ctypes.POINTER(ctypes.c_int)], ctypes.c_int),
    "lego_layout_dims": ([_vp, ctypes.c_int, c_i64p], ctypes.c_int),
    "lego_layout_size": ([_vp, c_i64p], ctypes.c_int),
    "lego_layout_phys_size": ([_vp, c_i64p], ctypes.c_int),
    "lego_apply": ([_vp, c_i64p, c_i64p], ctypes.c_int),
    "lego_inv": ([_vp, ctypes.c_int64, c_i64p], ctypes.c_int),
    "lego_verify_bijective": ([_vp, ctypes.c_int64], ctypes.c_int),
    "lego_emit": ([_vp, ctypes.c_int, ctypes.c_char_p, ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)],
                  ctypes.c_int),
    "lego_apply_all_device": ([_vp, ctypes.c_int, _vp, _vp], ctypes.c_int),
    "lego_inv_all_device": ([_vp, ctypes.c_int, _vp, _vp], ctypes.c_int),
    "lego_remap": ([_vp, _vp, ctypes.c_int, _vp, _vp, _vp], ctypes.c_int),
    "lego_remap_plan": ([_vp, _vp, ctypes.c_int, ctypes.POINTER(ctypes.c_int), c_i64p, ctypes.POINTER(ctypes.c_int),
                         c_i64p, ctypes.c_char_p, ctypes.c_size_t], ctypes.c_int),
    "lego_gemm": ([ctypes.POINTER(lego_gemm_desc), _vp, _vp, _vp, _vp], ctypes.c_int),
    "lego_gemm_plan": ([ctypes.POINTER(lego_gemm_desc), ctypes.c_char_p, ctypes.c_size_t], ctypes.c_int),
    "lego_mfma_fragment_layout": ([ctypes.c_int, ctypes.c_int, ctypes.POINTER(_vp)], ctypes.c_int),
    "lego_selftest_compile": ([ctypes.POINTER(ctypes.c_int), ctypes.c_char_p, ctypes.c_size_t], ctypes.c_int),
    "lego_plan_source": ([ctypes.c_int, _vp, _vp, ctypes.c_int, ctypes.POINTER(lego_gemm_desc), ctypes.c_char_p,
                          ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
    "lego_selftest_source": ([ctypes.c_int, ctypes.c_char_p, ctypes.c_size_t, ctypes.c_char_p, ctypes.c_size_t,
                              ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
}
for _name, (_args, _res) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res
    globals()[_name] = _f

EXPORTED = tuple(_SIGS)


def _check(rc):
    if rc != LEGO_OK:
        raise LegoError(rc, _lib.lego_last_error().decode())
    return rc


def _i64(xs):
    xs = [int(x) for x in xs]
    return (ctypes.c_int64 * max(1, len(xs)))(*xs)


_RAW_STREAM = None


def _current_stream():
    """torch's current HIP stream on the current device (the raw lookup costs
    a fraction of a microsecond; torch.cuda.current_stream() several)."""
    global _RAW_STREAM
    if _RAW_STREAM is None:
        import torch
        get, dev = getattr(torch._C, "_cuda_getCurrentRawStream", None), getattr(torch._C, "_cuda_getDevice", None)
        if get is not None and dev is not None:
            _RAW_STREAM = lambda: get(dev())  # noqa: E731
        else:
            _RAW_STREAM = lambda: torch.cuda.current_stream().cuda_stream  # noqa: E731
    return _RAW_STREAM()


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(_current_stream())
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


class _Handle:
    __slots__ = ("h",)

    def __init__(self, h):
        self.h = ctypes.c_void_p(h) if not isinstance(h, ctypes.c_void_p) else h

    def __del__(self):
        try:
            if self.h and _lib is not None:
                _lib.lego_release(self.h)
                self.h = None
        except Exception:
            pass


class Piece(_Handle):
    """A RegP or GenP permutation of one tile (Figure 3)."""

    def dims(self):
        r = ctypes.c_int()
        d = (ctypes.c_int64 * 16)()
        _check(_lib.lego_piece_dims(self.h, ctypes.byref(r), d))
        return list(d[:r.value])


def RegP(dims, sigma):  # noqa: N802 (paper notation)
    if len(sigma) != len(dims):
        # the C call reads len(dims) permutation entries
        raise LegoError(-1, "sigma must have one entry per tile dimension")
    out = ctypes.c_void_p()
    s = (ctypes.c_int32 * len(sigma))(*[int(x) for x in sigma])
    _check(_lib.lego_regp(len(dims), _i64(dims), s, ctypes.byref(out)))
    return Piece(out)


def Row(*dims):  # noqa: N802
    dims = _dims(dims)
    out = ctypes.c_void_p()
    _check(_lib.lego_row(len(dims), _i64(dims), ctypes.byref(out)))
    return Piece(out)


def Col(*dims):  # noqa: N802
    dims = _dims(dims)
    out = ctypes.c_void_p()
    _check(_lib.lego_col(len(dims), _i64(dims), ctypes.byref(out)))
    return Piece(out)


def GenP(kind, dims, params=()):  # noqa: N802
    out = ctypes.c_void_p()
    k = GENP[kind] if isinstance(kind, str) else int(kind)
    _check(_lib.lego_genp(k, len(dims), _i64(dims), _i64(params), len(params), ctypes.byref(out)))
    return Piece(out)


def GenPExpr(dims, apply, inv):  # noqa: N802
    """A user-defined GenP from integer expressions (grammar in include/lego.h):
    ``apply`` over i0..i{d-1} (or i, j, k), ``inv`` one expression per
    dimension over x."""
    if isinstance(inv, str) or len(inv) != len(dims):
        raise LegoError(-1, "inv must hold one expression per dimension")
    if any(";" in t for t in inv):
        raise LegoError(-1, "';' separates the inverse expressions")
    out = ctypes.c_void_p()
    _check(_lib.lego_genp_expr(len(dims), _i64(dims), apply.encode(), ";".join(inv).encode(), ctypes.byref(out)))
    return Piece(out)


def _dims(d):
    if len(d) == 1 and isinstance(d[0], (list, tuple)):
        return [int(x) for x in d[0]]
    return [int(x) for x in d]


class Layout(_Handle):
    """A GroupBy chain (Figure 5); ``.OrderBy`` appends in dot notation."""

    def OrderBy(self, *pieces):  # noqa: N802
        arr = (ctypes.c_void_p * len(pieces))(*[p.h for p in pieces])
        out = ctypes.c_void_p()
        _check(_lib.lego_orderby(self.h, len(pieces), arr, ctypes.byref(out)))
        return Layout(out)

    def rank(self):
        r = ctypes.c_int()
        _check(_lib.lego_layout_rank(self.h, ctypes.byref(r)))
        return r.value

    def dims(self):
        n = self.rank()
        d = (ctypes.c_int64 * n)()
        _check(_lib.lego_layout_dims(self.h, n, d))
        return list(d)

    def size(self):
        n = ctypes.c_int64()
        _check(_lib.lego_layout_size(self.h, ctypes.byref(n)))
        return n.value

    def phys_size(self):
        """Elements of a buffer in this layout (ExpandBy: the original extents)."""
        n = ctypes.c_int64()
        _check(_lib.lego_layout_phys_size(self.h, ctypes.byref(n)))
        return n.value

    def apply(self, idx):
        if len(idx) != self.rank():
            raise LegoError(-1, "index rank differs from the layout rank")
        f = ctypes.c_int64()
        _check(_lib.lego_apply(self.h, _i64(idx), ctypes.byref(f)))
        return f.value

    def inv(self, flat):
        n = self.rank()
        d = (ctypes.c_int64 * n)()
        _check(_lib.lego_inv(self.h, int(flat), d))
        return list(d)

    def verify_bijective(self, max_points=1 << 24):
        _check(_lib.lego_verify_bijective(self.h, int(max_points)))
        return True

    def emit(self, which="apply"):
        need = ctypes.c_size_t()
        w = 0 if which == "apply" else 1
        _check(_lib.lego_emit(self.h, w, None, 0, ctypes.byref(need)))
        buf = ctypes.create_string_buffer(need.value)
        _check(_lib.lego_emit(self.h, w, buf, need.value, ctypes.byref(need)))
        return buf.value.decode()


def GroupBy(*tiles):  # noqa: N802
    dims = [int(x) for t in tiles for x in (t if isinstance(t, (list, tuple)) else [t])]
    out = ctypes.c_void_p()
    _check(_lib.lego_groupby(len(dims), _i64(dims), ctypes.byref(out)))
    return Layout(out)


def GroupByTiles(*tiles):  # noqa: N802
    """GroupBy over q tile levels of equal rank d (lego_groupby_tiles)."""
    q, d = len(tiles), len(tiles[0])
    flat = [int(x) for t in tiles for x in t]
    if any(len(t) != d for t in tiles):
        raise LegoError(-1, "GroupBy tile levels must have equal rank")
    out = ctypes.c_void_p()
    _check(_lib.lego_groupby_tiles(q, d, _i64(flat), ctypes.byref(out)))
    return Layout(out)


def TileBy(*tiles):  # noqa: N802
    q, d = len(tiles), len(tiles[0])
    if any(len(t) != d for t in tiles):
        raise LegoError(-1, "TileBy levels must have equal rank")
    flat = [int(x) for t in tiles for x in t]
    out = ctypes.c_void_p()
    _check(_lib.lego_tileby(q, d, _i64(flat), ctypes.byref(out)))
    return Layout(out)


def TileOrderBy(*pieces):  # noqa: N802
    arr = (ctypes.c_void_p * len(pieces))(*[p.h for p in pieces])
    out = ctypes.c_void_p()
    _check(_lib.lego_tileorderby(len(pieces), len(pieces[0].dims()), arr, ctypes.byref(out)))
    return Layout(out)


def _tileorderby_d(d, *pieces):
    """lego_tileorderby with an explicit level rank d (tests of its check)."""
    arr = (ctypes.c_void_p * len(pieces))(*[p.h for p in pieces])
    out = ctypes.c_void_p()
    _check(_lib.lego_tileorderby(len(pieces), int(d), arr, ctypes.byref(out)))
    return Layout(out)


def as_layout(piece):
    out = ctypes.c_void_p()
    _check(_lib.lego_layout_from_piece(piece.h, ctypes.byref(out)))
    return Layout(out)


def ExpandBy(n, n_expanded, g):  # noqa: N802
    if len(n) != len(n_expanded):
        raise LegoError(-1, "ExpandBy extents must have equal rank")
    out = ctypes.c_void_p()
    _check(_lib.lego_expandby(len(n), _i64(n), _i64(n_expanded), g.h, ctypes.byref(out)))
    return Layout(out)


def mfma_fragment_layout(instr, operand):
    out = ctypes.c_void_p()
    _check(_lib.lego_mfma_fragment_layout(int(instr), int(operand), ctypes.byref(out)))
    return Layout(out)


# ------------------------------------------------------------------ device --
def apply_all_device(layout, out, stream=None):
    """out[x] = apply(x) for every logical flat x (out: int32/int64 cuda tensor)."""
    _need(out, layout.size(), "output")
    _check(_lib.lego_apply_all_device(layout.h, out.element_size(), _ptr(out), _stream(stream)))


def inv_all_device(layout, out, stream=None):
    """out[p, k] = inv(p)[k] for every physical p (out: [N, rank] int32/int64)."""
    _need(out, layout.phys_size() * layout.rank(), "output")
    _check(_lib.lego_inv_all_device(layout.h, out.element_size(), _ptr(out), _stream(stream)))


def _need(t, n, what):
    # the kernels index up to n elements of the buffer
    if t.numel() < n:
        raise LegoError(-2, f"{what} holds {t.numel()} elements, the layout needs {n}")


def remap(src_layout, dst_layout, src, dst, stream=None):
    """dst[dst.apply(x)] = src[src.apply(x)] for all logical x (cuda tensors);
    positions of dst outside an ExpandBy source's extents become zero."""
    if src.element_size() != dst.element_size():
        raise LegoError(-1, "source and destination element sizes differ")
    _need(src, src_layout.phys_size(), "source")
    _need(dst, dst_layout.phys_size(), "destination")
    _check(_lib.lego_remap(src_layout.h, dst_layout.h, src.element_size(), _ptr(src), _ptr(dst), _stream(stream)))


def remap_plan(src_layout, dst_layout, elem_bytes):
    path, vec = ctypes.c_int(), ctypes.c_int()
    run, tile = ctypes.c_int64(), ctypes.c_int64()
    info = ctypes.create_string_buffer(4096)
    _check(_lib.lego_remap_plan(src_layout.h, dst_layout.h, int(elem_bytes), ctypes.byref(path), ctypes.byref(run),
                                ctypes.byref(vec), ctypes.byref(tile), info, 4096))
    return {"path": ("direct", "lds", "gather", "box")[path.value], "run": run.value, "vec": vec.value,
            "tile": tile.value, "info": info.value.decode()}


def _desc(M, N, K, dtype, a=None, b=None, c=None, sched=None, lds_a=None, lds_b=None, bm=0, bn=0, bk=0, wm=0, wn=0,
          group_m=0, xcd_remap=1, stages=0, max_workgroups=0, frag_a=None, frag_b=None, frag_c=None):
    d = lego_gemm_desc()
    d.M, d.N, d.K = int(M), int(N), int(K)
    d.in_dtype = DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
    d.bm, d.bn, d.bk, d.wm, d.wn, d.group_m, d.xcd_remap = bm, bn, bk, wm, wn, group_m, xcd_remap
    d.stages = stages
    d.max_workgroups = max_workgroups
    for name, lay in (("a", a), ("b", b), ("c", c), ("sched", sched), ("lds_a", lds_a), ("lds_b", lds_b),
                      ("frag_a", frag_a), ("frag_b", frag_b), ("frag_c", frag_c)):
        setattr(d, name, lay.h if lay is not None else None)
    return d


def gemm(A, B, C, M, N, K, dtype, stream=None, **kw):
    """C (fp32) = A @ B with operands in their layouts (cuda tensors)."""
    for t, lay, n, what in ((A, kw.get("a"), M * K, "A"), (B, kw.get("b"), K * N, "B"), (C, kw.get("c"), M * N, "C")):
        _need(t, lay.phys_size() if lay is not None else n, what)
    d = _desc(M, N, K, dtype, **kw)
    _check(_lib.lego_gemm(ctypes.byref(d), _ptr(A), _ptr(B), _ptr(C), _stream(stream)))


def gemm_plan(M, N, K, dtype, **kw):
    d = _desc(M, N, K, dtype, **kw)
    info = ctypes.create_string_buffer(8192)
    _check(_lib.lego_gemm_plan(ctypes.byref(d), info, 8192))
    return info.value.decode()


def selftest_compile():
    n = ctypes.c_int()
    info = ctypes.create_string_buffer(1 << 16)
    _check(_lib.lego_selftest_compile(ctypes.byref(n), info, 1 << 16))
    return n.value, info.value.decode()


def plan_source(kind, x=None, y=None, param=0, **gemm_kw):
    """Generated source of a plan: kind 'apply'/'inv' of layout x (param =
    idx_bytes), 'remap' from layout x to layout y (param = elem_bytes) or
    'gemm' (gemm_kw as for gemm(), operand layouts included)."""
    k = {"apply": 0, "inv": 1, "remap": 2, "gemm": 3}[kind]
    if k != 3 and gemm_kw:
        raise TypeError(f"unexpected arguments for '{kind}': {sorted(gemm_kw)}")
    d = ctypes.byref(_desc(**gemm_kw)) if k == 3 else None
    need = ctypes.c_size_t()
    ah = x.h if x is not None else None
    bh = y.h if y is not None else None
    _check(_lib.lego_plan_source(k, ah, bh, int(param), d, None, 0, ctypes.byref(need)))
    buf = ctypes.create_string_buffer(need.value)
    _check(_lib.lego_plan_source(k, ah, bh, int(param), d, buf, need.value, ctypes.byref(need)))
    return buf.value.decode()


def selftest_sources():
    """[(name, generated source)] of the built-in configurations."""
    out = []
    i = 0
    while True:
        need = ctypes.c_size_t()
        name = ctypes.create_string_buffer(256)
        rc = _lib.lego_selftest_source(i, name, 256, None, 0, ctypes.byref(need))
        if rc != LEGO_OK:
            break
        buf = ctypes.create_string_buffer(need.value)
        _check(_lib.lego_selftest_source(i, name, 256, buf, need.value, ctypes.byref(need)))
        out.append((name.value.decode(), buf.value.decode()))
        i += 1
    return out


def library_path():
    return _LIBPATH
