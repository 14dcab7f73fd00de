"""CPU oracle for layout-mapped data movement (LEGO, arXiv 2505.08091).

TEST INFRASTRUCTURE ONLY.  Nothing in the product package may import, call or
execute anything in this directory; only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.

The oracle is deliberately plain and slow: layouts are evaluated point by point
following the paper's definitions (Section III-B, Figures 3, 4 and 5), remaps
are per-point copies, and the GEMM is an fp64 product of the exactly decoded
fp16/bf16 inputs.  It shares no code with the HIP path.  Every function cites
the passage it follows; readings of ambiguous passages are listed in the
module docstrings where they are used.

Modules
  layout  canonical bijections, RegP, GenP, OrderBy, GroupBy, ExpandBy, sugar,
          and the named irregular permutations (reverse, antidiagonal,
          Morton, XOR swizzle).
  remap   the permutation dst[L_dst.apply(x)] = src[L_src.apply(x)].
  gemm    C = A @ B in fp64 with operands read through layouts.
  genexpr user-defined GenP pieces written as integer expressions.
"""
from . import layout, remap, gemm, genexpr  # noqa: F401
