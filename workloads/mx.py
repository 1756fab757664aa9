"""Seeded inputs for the block-scaled minifloat matmul (ScaledMatMul).

Draws element codes and E8M0 block scales directly -- no quantiser: the op's
inputs are codes, so random finite codes with the format's bit width are a
complete input distribution.  Holds none of the op's arithmetic: codes are
drawn as integers and only laid out into the storage format (FP8 one byte per
code, FP4 two per byte with the lower k in the low nibble, FP6 four codes per
three bytes as a little-endian bit stream).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

BLOCK = 32
BITS = {"e4m3": 8, "e5m2": 8, "e2m3": 6, "e3m2": 6, "e2m1": 4}
# codes that are NaN or Inf in their format (drawn codes avoid them)
_SPECIAL = {"e4m3": {0x7F, 0xFF}, "e5m2": set(range(0x7C, 0x80)) | set(range(0xFC, 0x100))}


def finite_codes(fmt: str) -> np.ndarray:
    bits = BITS[fmt]
    return np.array([c for c in range(1 << bits) if c not in _SPECIAL.get(fmt, set())], dtype=np.uint8)


def pack(codes: np.ndarray, fmt: str) -> np.ndarray:
    """Codes [R, K] -> stored rows."""
    q = np.asarray(codes, dtype=np.uint8)
    R, K = q.shape
    bits = BITS[fmt]
    if bits == 8:
        return q.copy()
    if bits == 4:
        return (q[:, 0::2] | (q[:, 1::2] << 4)).astype(np.uint8)
    g = q.reshape(R, K // 4, 4).astype(np.uint32)
    word = g[:, :, 0] | (g[:, :, 1] << 6) | (g[:, :, 2] << 12) | (g[:, :, 3] << 18)
    out = np.stack([word & 0xFF, (word >> 8) & 0xFF, (word >> 16) & 0xFF], axis=-1)
    return out.reshape(R, K * 3 // 4).astype(np.uint8)


@dataclass
class MxOperand:
    fmt: str
    codes: np.ndarray    # [R, K] uint8
    packed: np.ndarray   # stored rows
    scales: np.ndarray   # [R, K/32] uint8 (E8M0)


def operand(rng: np.random.Generator, rows: int, K: int, fmt: str, scale_lo: int = 120, scale_hi: int = 134,
            allowed_codes=None) -> MxOperand:
    """Uniform draws over ``allowed_codes`` (default: every finite code) and
    scales uniform in [scale_lo, scale_hi]."""
    assert K % BLOCK == 0
    pool = finite_codes(fmt) if allowed_codes is None else np.asarray(allowed_codes, dtype=np.uint8)
    codes = pool[rng.integers(0, len(pool), size=(rows, K))]
    scales = rng.integers(scale_lo, scale_hi + 1, size=(rows, K // BLOCK)).astype(np.uint8)
    return MxOperand(fmt, codes, pack(codes, fmt), scales)


def exact_codes(fmt: str) -> np.ndarray:
    """Codes whose products and float32 partial sums stay exact in the tests
    that compare bit for bit (K <= 512, scales 2^-1 .. 2^1): zero and the
    values within one binade of 1 (the [1, 2) binade alone for the formats
    with three mantissa bits)."""
    bits = BITS[fmt]
    e_bits, bias = {"e4m3": (4, 7), "e5m2": (5, 15), "e2m3": (2, 1), "e3m2": (3, 3), "e2m1": (2, 1)}[fmt]
    m_bits = bits - 1 - e_bits
    reach = 0 if m_bits == 3 else 1
    keep = []
    for c in finite_codes(fmt):
        e = (int(c) >> m_bits) & ((1 << e_bits) - 1)
        if (int(c) & ((1 << (bits - 1)) - 1)) == 0 or abs(e - bias) <= reach:
            keep.append(c)
    return np.array(keep, dtype=np.uint8)


def matmul_inputs(seed: int, M: int, N: int, K: int, fa: str, fb: str, exact: bool = False):
    """A [M, K] and B [N, K] operands; ``exact`` narrows codes and scales so that
    every float32 partial sum of the product is exact (bit-exact comparisons)."""
    rng = np.random.default_rng(seed)
    if exact:
        a = operand(rng, M, K, fa, 126, 128, exact_codes(fa))
        b = operand(rng, N, K, fb, 126, 128, exact_codes(fb))
    else:
        a = operand(rng, M, K, fa)
        b = operand(rng, N, K, fb)
    return a, b
