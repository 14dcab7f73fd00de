"""Oracle: user-defined GenP pieces written as integer expressions.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Section III-B allows a GenP to be any bijection f of a tile with its inverse.
The library accepts f and f^-1 as text in a small C-like integer language;
this module evaluates the same language independently, on Python ints and,
elementwise, on numpy int64 arrays:

* integers; the coordinates ``i0 .. i{d-1}`` (``i``, ``j``, ``k`` for the
  first three) in f, ``x`` in f^-1, the tile extents ``n0 .. n{d-1}``;
* ``+ - *``, floor ``/`` and ``%``, ``<< >>``, ``&`` (with a mask 2^k - 1),
  ``^``, comparisons ``< <= > >= == !=`` giving 0/1, ``!``, ``&&``, ``||``,
  ``c ? a : b``, parentheses, ``isqrt`` (exact floor square root), ``min``,
  ``max``, with C's operator precedence.

The forward result is taken modulo the tile size and inverse coordinate k
modulo extent n_k (the identity for a bijection onto the tile).
"""
from __future__ import annotations

import math
import re

import numpy as np

from .layout import GenP

_TOKEN = re.compile(r"\s*(?:(\d+)|([A-Za-z_]\w*)|(<<|>>|<=|>=|==|!=|&&|\|\||[-+*/%^&<>!?:(),]))")


def _tokens(text):
    pos, out = 0, []
    text = text.rstrip()
    while pos < len(text):
        m = _TOKEN.match(text, pos)
        if not m or m.end() == pos:
            raise ValueError(f"bad character at offset {pos} of {text!r}")
        out.append(("num", int(m.group(1))) if m.group(1) else ("name", m.group(2)) if m.group(2) else ("op", m.group(3)))
        pos = m.end()
    return out


def _isqrt(v):
    if isinstance(v, np.ndarray):
        return np.array([math.isqrt(int(t)) for t in v.ravel()], dtype=np.int64).reshape(v.shape)
    return math.isqrt(int(v))


def _b(v):
    """0/1 of a truth value (array or scalar)."""
    if isinstance(v, np.ndarray):
        return v.astype(np.int64)
    return int(bool(v))


def _where(c, a, b):
    if isinstance(c, np.ndarray) or isinstance(a, np.ndarray) or isinstance(b, np.ndarray):
        return np.where(np.asarray(c) != 0, a, b)
    return a if c else b


# binary operators by C precedence level (higher binds tighter)
_BIN = {
    "||": (1, lambda a, b: _b((a != 0) | (b != 0)) if isinstance(a, np.ndarray) or isinstance(b, np.ndarray)
           else int(bool(a) or bool(b))),
    "&&": (2, lambda a, b: _b((a != 0) & (b != 0)) if isinstance(a, np.ndarray) or isinstance(b, np.ndarray)
           else int(bool(a) and bool(b))),
    "^": (3, lambda a, b: a ^ b),
    "&": (4, lambda a, b: a & b),
    "==": (5, lambda a, b: _b(a == b)),
    "!=": (5, lambda a, b: _b(a != b)),
    "<": (6, lambda a, b: _b(a < b)),
    "<=": (6, lambda a, b: _b(a <= b)),
    ">": (6, lambda a, b: _b(a > b)),
    ">=": (6, lambda a, b: _b(a >= b)),
    "<<": (7, lambda a, b: a * (1 << b)),
    ">>": (7, lambda a, b: a // (1 << b)),
    "+": (8, lambda a, b: a + b),
    "-": (8, lambda a, b: a - b),
    "*": (9, lambda a, b: a * b),
    "/": (9, lambda a, b: a // b),
    "%": (9, lambda a, b: a % b),
}


class _Parser:
    """Precedence climbing over the token list; builds a closure env -> value."""

    def __init__(self, text, names):
        self.t = _tokens(text)
        self.p = 0
        self.names = names
        self.text = text

    def peek(self):
        return self.t[self.p] if self.p < len(self.t) else ("end", None)

    def take(self, op):
        if self.peek() == ("op", op):
            self.p += 1
            return True
        return False

    def parse(self):
        e = self.cond()
        if self.p != len(self.t):
            raise ValueError(f"trailing text in {self.text!r}")
        return e

    def cond(self):
        c = self.binary(1)
        if self.take("?"):
            a = self.cond()
            if not self.take(":"):
                raise ValueError(f"expected ':' in {self.text!r}")
            b = self.cond()
            return lambda env: _where(c(env), a(env), b(env))
        return c

    def binary(self, level):
        lhs = self.unary()
        while True:
            kind, op = self.peek()
            if kind != "op" or op not in _BIN or _BIN[op][0] < level:
                return lhs
            prec, fn = _BIN[op]
            self.p += 1
            rhs = self.binary(prec + 1)
            lhs = (lambda f, a, b: lambda env: f(a(env), b(env)))(fn, lhs, rhs)

    def unary(self):
        if self.take("-"):
            a = self.unary()
            return lambda env: -a(env)
        if self.take("!"):
            a = self.unary()
            return lambda env: _b(a(env) == 0)
        return self.primary()

    def primary(self):
        kind, v = self.peek()
        self.p += 1
        if kind == "num":
            return lambda env: v
        if kind == "op" and v == "(":
            e = self.cond()
            if not self.take(")"):
                raise ValueError(f"expected ')' in {self.text!r}")
            return e
        if kind == "name":
            if v in ("isqrt", "min", "max"):
                if not self.take("("):
                    raise ValueError(f"expected '(' after {v}")
                args = [self.cond()]
                while self.take(","):
                    args.append(self.cond())
                if not self.take(")"):
                    raise ValueError(f"expected ')' in {self.text!r}")
                if v == "isqrt":
                    a = args[0]
                    return lambda env: _isqrt(a(env))
                a, b = args
                if v == "min":
                    return lambda env: np.minimum(a(env), b(env)) if isinstance(a(env), np.ndarray) else min(a(env), b(env))
                return lambda env: np.maximum(a(env), b(env)) if isinstance(a(env), np.ndarray) else max(a(env), b(env))
            if v not in self.names:
                raise ValueError(f"unknown name {v!r} in {self.text!r}")
            return lambda env: env[v]
        raise ValueError(f"unexpected token {v!r} in {self.text!r}")


def evaluate(text, **env):
    """Value of one expression with the given names bound (ints or arrays)."""
    return _Parser(text, set(env)).parse()(env)


def expr_genp(dims, apply_src, inv_srcs):
    """GenP over ``dims`` from the forward expression and one inverse
    expression per dimension."""
    dims = [int(x) for x in dims]
    d = len(dims)
    consts = {f"n{k}": dims[k] for k in range(d)}
    fwd_names = set(consts) | {f"i{k}" for k in range(d)} | {"ijk"[k] for k in range(min(d, 3))}
    f = _Parser(apply_src, fwd_names).parse()
    g = [_Parser(s, set(consts) | {"x"}).parse() for s in inv_srcs]
    if len(g) != d:
        raise ValueError("one inverse expression per dimension")

    size = 1
    for v in dims:
        size *= v

    def fwd(*i):
        env = dict(consts)
        for k in range(d):
            env[f"i{k}"] = i[k]
            if k < 3:
                env["ijk"[k]] = i[k]
        return f(env) % size  # results are defined modulo the tile size

    def inv(x):
        env = dict(consts)
        env["x"] = x
        return [h(env) % dims[k] for k, h in enumerate(g)]  # and modulo each extent

    return GenP(dims, fwd, inv, name="expr")
