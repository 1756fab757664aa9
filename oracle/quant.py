"""Weight-only dequantisation (test infrastructure; see package docstring).

The paper's Op::DequantMatMul (Sections III-A and VI) multiplies activations by
weights stored in a quantised scheme and dequantised on the fly; it names the
llama.cpp scheme family from INT8 to INT4 (Section III-B, numeric precision)
without fixing a layout.  Readings taken here:

* int8: symmetric, one fp16 scale per output channel n:  W[n,k] = q[n,k] * s[n].
* int4: unsigned codes 0..15 with one fp16 scale and one fp16 integer-valued
  zero-point per group of ``group`` consecutive k:  W[n,k] = (q[n,k] - z[n,g]) * s[n,g],
  g = k // group.  Two codes per byte: byte j of a row holds k = 2j in its low
  nibble and k = 2j+1 in its high nibble.

Both products are exact in float32 (and float64).
"""
from __future__ import annotations

import numpy as np


def unpack_int4(packed):
    """[N, K/2] bytes -> [N, K] codes 0..15 (low nibble first)."""
    p = np.asarray(packed, dtype=np.uint8)
    n, kh = p.shape
    q = np.empty((n, 2 * kh), dtype=np.uint8)
    q[:, 0::2] = p & 0x0F
    q[:, 1::2] = p >> 4
    return q


def dequant_int8(q, scales):
    """W = q * s per output channel; returns float64 [N, K]."""
    q = np.asarray(q, dtype=np.int8).astype(np.float64)
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    return q * s[:, None]


def dequant_int4(packed, scales, zeros, group):
    """W = (q - z) * s per group along K; returns float64 [N, K]."""
    q = unpack_int4(packed).astype(np.float64)
    n, k = q.shape
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    z = np.asarray(zeros, dtype=np.float16).astype(np.float64)
    assert s.shape == (n, k // group) and z.shape == s.shape
    g = np.arange(k) // group
    return (q - z[:, g]) * s[:, g]
