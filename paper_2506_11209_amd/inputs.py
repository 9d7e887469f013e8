"""Seeded synthetic operands for the GEMM workloads.

This module draws random numbers and rounds them to the 16-bit input format;
it performs none of the matrix product.  It is the one piece shared by the
oracle-based tests and the GPU path: both consume exactly the bit patterns
produced here.

All draws use torch's CPU generator (seeded), A first and then B, in float32,
followed by round-to-nearest-even into fp16 or bf16.
"""
from __future__ import annotations

import math

import numpy as np
import torch

TORCH_DTYPES = {"f16": torch.float16, "bf16": torch.bfloat16}
OUT_DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}

# value distributions
#   int4      integers uniform on {-4, ..., 4} (inclusive)
#   normal    i.i.d. N(0, 1)
#   uniform   i.i.d. U(-1, 1)
#   normal_k  i.i.d. N(0, 1) / sqrt(K)   (standard deviation 1/sqrt(K))
DISTRIBUTIONS = ("int4", "normal", "uniform", "normal_k")


def _draw(rows: int, cols: int, dist: str, K: int, g: torch.Generator) -> torch.Tensor:
    shape = (rows, cols)
    if dist == "int4":
        return torch.randint(-4, 5, shape, generator=g).to(torch.float32)
    if dist == "normal":
        return torch.randn(shape, generator=g)
    if dist == "uniform":
        return torch.rand(shape, generator=g) * 2.0 - 1.0
    if dist == "normal_k":
        return torch.randn(shape, generator=g) / math.sqrt(K)
    raise ValueError("unknown distribution %r" % dist)


def make_operands(M: int, N: int, K: int, dtype: str, dist: str, seed: int):
    """Return (A, B) as CPU tensors of the 16-bit dtype: A is M x K, B is K x N, row-major."""
    if dtype not in TORCH_DTYPES:
        raise ValueError("dtype must be one of %s" % list(TORCH_DTYPES))
    g = torch.Generator().manual_seed(seed)
    A = _draw(M, K, dist, K, g).to(TORCH_DTYPES[dtype]).contiguous()
    B = _draw(K, N, dist, K, g).to(TORCH_DTYPES[dtype]).contiguous()
    return A, B


def make_output(M: int, N: int, out_dtype: str, dist: str, seed: int) -> torch.Tensor:
    """The old C read by a beta != 0 epilogue: an M x N CPU tensor of the
    output type (f32, bf16 or f16), drawn like the operands (K = N for
    normal_k) and rounded to nearest even."""
    g = torch.Generator().manual_seed(seed)
    return _draw(M, N, dist, N, g).to(OUT_DTYPES[out_dtype]).contiguous()


def bits(t: torch.Tensor) -> np.ndarray:
    """The uint16 bit patterns of a 16-bit CPU tensor (shares memory)."""
    if t.dtype not in (torch.float16, torch.bfloat16):
        raise TypeError("expected an fp16/bf16 tensor")
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def from_bits(b: np.ndarray, dtype: str) -> torch.Tensor:
    """A CPU tensor of the 16-bit dtype holding the given bit patterns."""
    a = np.ascontiguousarray(b, dtype=np.uint16)
    return torch.from_numpy(a.view(np.int16)).view(TORCH_DTYPES[dtype])
