"""Seeded synthetic inputs shared by the oracle checks, the GPU tests and the
benchmark.

This module only draws numbers.  It holds none of the attention arithmetic and
none of the decomposition logic: it produces

* bf16 tensors of i.i.d. N(0, 1) values (numpy ``default_rng``, float32 draws
  rounded to bf16 with round-to-nearest-even), returned as uint16 bit patterns
  so that the oracle and the GPU see the same bytes;
* document lengths for the concat-and-chunk workload: a log-normal stand-in for
  the web-crawl length distribution the paper trains on (its figures give the
  shape only), median 600 tokens, sigma 1.2, clipped to [1, 8192], drawn until
  the step's token budget is filled and the last document truncated;
* the per-step sequence lengths of a short-biased length stream, with weights
  proportional to 1/L (the odds of the paper's "Grow-P2" curriculum, drawn
  i.i.d. here).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "bf16_bits_from_f32",
    "f32_from_bf16_bits",
    "normal_bf16",
    "attention_inputs",
    "lognormal_doc_lengths",
    "length_stream",
]

# Stream ids for the four attention operands, so each draws its own numbers.
_STREAM = {"q": 1, "k": 2, "v": 3, "do": 4}


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even).

    Returns the uint16 bit patterns.  NaN inputs stay NaN (quiet bit set).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    bits = rounded.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        bits[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return bits


def f32_from_bf16_bits(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def normal_bf16(shape, seed: int, stream: int = 0) -> np.ndarray:
    """i.i.d. N(0, 1) values rounded to bf16, as uint16 bits of ``shape``."""
    rng = np.random.default_rng([int(seed), int(stream)])
    x = rng.standard_normal(size=int(np.prod(shape)), dtype=np.float32)
    return bf16_bits_from_f32(x).reshape(shape)


def attention_inputs(B: int, L: int, H: int, D: int, seed: int = 0,
                     with_grad: bool = True) -> dict:
    """Q, K, V (and the upstream gradient dO) as bf16 bits, each [B, L, H, D]."""
    names = ["q", "k", "v"] + (["do"] if with_grad else [])
    return {n: normal_bf16((B, L, H, D), seed, _STREAM[n]) for n in names}


def lognormal_doc_lengths(seed: int, total_tokens: int = 65536,
                          median: float = 600.0, sigma: float = 1.2,
                          max_len: int = 8192) -> np.ndarray:
    """Document lengths whose sum is exactly ``total_tokens``.

    Each length is rint(exp(N(ln median, sigma^2))) clipped to [1, max_len];
    lengths are drawn in order until the running sum reaches the budget and the
    last one is cut so the sum is exact.  Draw order is concatenation order.
    """
    rng = np.random.default_rng(int(seed))
    out = []
    acc = 0
    while acc < total_tokens:
        ell = int(np.clip(np.rint(np.exp(rng.normal(np.log(median), sigma))),
                          1, max_len))
        ell = min(ell, total_tokens - acc)
        out.append(ell)
        acc += ell
    return np.asarray(out, dtype=np.int64)


def length_stream(seed: int, steps: int = 64,
                  lengths=(256, 512, 1024, 2048, 4096, 8192, 16384)) -> np.ndarray:
    """Sequence length of each step, drawn i.i.d. with weights 1/L."""
    rng = np.random.default_rng(int(seed))
    lens = np.asarray(lengths, dtype=np.int64)
    w = 1.0 / lens.astype(np.float64)
    return rng.choice(lens, size=int(steps), p=w / w.sum())
