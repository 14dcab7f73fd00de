"""Seeded synthetic inputs shared by the tests, the bench and the oracle.

This module holds no layout or GEMM arithmetic: it only draws numbers.  Values
are generated in fp32 by a CPU ``torch.Generator`` seeded with ``seed`` and
cast once with round-to-nearest-even to the requested element type, so the GPU
path and the oracle consume exactly the same bytes.

Workload recipe (synthetic stand-ins for the paper's square power-of-two
matrices, Section V):
  * "uniform": U[-1, 1)  (``rand * 2 - 1``)
  * "normal":  N(0, 1)   (``randn``)
  * "smallint": integers in {-2, ..., 2}, exactly representable in fp16/bf16,
    used for the exactly-checkable GEMM case.
Seeds: A = 1, B = 2, remap source = 3.
"""
from __future__ import annotations

import numpy as np
import torch

SEED_A = 1
SEED_B = 2
SEED_SRC = 3

_TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def tensor(n, dtype="f32", dist="uniform", seed=SEED_SRC):
    """Flat CPU torch tensor of n elements of ``dtype`` ('f32', 'f16', 'bf16')."""
    g = torch.Generator().manual_seed(int(seed))
    if dist == "uniform":
        x = torch.rand(int(n), generator=g, dtype=torch.float32) * 2 - 1
    elif dist == "normal":
        x = torch.randn(int(n), generator=g, dtype=torch.float32)
    elif dist == "smallint":
        x = torch.randint(-2, 3, (int(n),), generator=g).to(torch.float32)
    elif dist == "iota":
        x = torch.arange(int(n), dtype=torch.float32)
    else:
        raise ValueError(dist)
    return x.to(_TORCH_DT[dtype])


def as_numpy_bits(t):
    """The raw bytes of a CPU tensor as a numpy array (uint16 for 2-byte types,
    float32 for f32), for the oracle."""
    if t.dtype in (torch.float16, torch.bfloat16):
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def int_tensor(n, seed=SEED_SRC, bits=32):
    """Flat CPU int32 tensor of distinct-looking values for bit-exact remap
    tests of 4-byte elements (a random permutation of arange(n))."""
    g = torch.Generator().manual_seed(int(seed))
    return torch.randperm(int(n), generator=g).to(torch.int32 if bits == 32 else torch.int64)


def _byte_hash(i, seed):
    """High byte of a 32-bit multiplicative hash of (index, seed); every
    intermediate stays below 2^63 so int64 arithmetic is exact."""
    lo, hi = i & 0xFFFFFFFF, i >> 32
    h = (lo * 0x5BD1E995 + hi * 0x1B873593 + int(seed) * 0x27D4EB2F) & 0xFFFFFFFF
    h = ((h ^ (h >> 15)) * 0x2C1B3C6D) & 0xFFFFFFFF
    return (h >> 24) & 255


def byte_pattern(start, count, seed=SEED_SRC, device="cpu"):
    """uint8 elements start .. start+count-1 of a pseudo-random byte array of
    any length (buffers beyond 2^32 elements are filled slice by slice, on
    the device that holds them)."""
    i = torch.arange(int(start), int(start) + int(count), dtype=torch.int64, device=device)
    return _byte_hash(i, seed).to(torch.uint8)


def byte_pattern_at(idx, seed=SEED_SRC):
    """The same bytes at the int64 numpy indices ``idx``."""
    return _byte_hash(np.asarray(idx, dtype=np.int64), seed).astype(np.uint8)
