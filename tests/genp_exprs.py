"""Expression GenPs used by the tests (the same text goes to the library and
to the oracle's independent evaluator)."""

# Figure 7's antidiagonal order as closed forms: the antidiagonal a = i + j
# holds a + 1 elements above the main antidiagonal (triangular numbers), and
# the lower half mirrors the upper one through x -> n^2 - 1 - x.
ANTIDIAG_APPLY = ("i + j < n0 ? i + (i + j) * (i + j + 1) / 2"
                  " : n0 * n0 - 1 - ((n0 - 1 - i) + (2 * n0 - 2 - i - j) * (2 * n0 - 1 - i - j) / 2)")
_T = "(isqrt(8 * {y} + 1) - 1) / 2"          # antidiagonal index of upper-half position y
_R = "({y} - {t} * ({t} + 1) / 2)"           # row within that antidiagonal
_UP = "x < n0 * (n0 + 1) / 2"
_Y = "(n0 * n0 - 1 - x)"


def _row(y):
    t = _T.format(y=y)
    return _R.format(y=y, t=t)


def _col(y):
    t = _T.format(y=y)
    return f"({t} - {_R.format(y=y, t=t)})"


ANTIDIAG_INV = [f"{_UP} ? {_row('x')} : n0 - 1 - {_row(_Y)}",
                f"{_UP} ? {_col('x')} : n0 - 1 - {_col(_Y)}"]

# Z order of an 8 x 8 tile: column bits at even, row bits at odd positions.
MORTON8_APPLY = ("(j & 1) + ((i & 1) << 1) + (((j >> 1) & 1) << 2) + (((i >> 1) & 1) << 3)"
                 " + (((j >> 2) & 1) << 4) + (((i >> 2) & 1) << 5)")
MORTON8_INV = ["((x >> 1) & 1) + (((x >> 3) & 1) << 1) + (((x >> 5) & 1) << 2)",
               "(x & 1) + (((x >> 2) & 1) << 1) + (((x >> 4) & 1) << 2)"]

# A user-written LDS swizzle for a [rows, 64] fp16 tile: 16-byte vectors of a
# row XOR-permuted by row / 2 (the built-in xor_swizzle with v = 8, s = 2).
SWIZZLE64_APPLY = "i * 64 + (((j / 8) ^ ((i / 2) % 8)) * 8) + j % 8"
SWIZZLE64_INV = ["x / 64", "(((x % 64) / 8) ^ ((x / 128) % 8)) * 8 + x % 8"]
