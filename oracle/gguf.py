"""GGUF weight blocks (test infrastructure; see package docstring).

The paper's Op::DequantMatMul covers the llama.cpp / GGUF scheme set
(Section VI, quantized inference: Q4_0 .. Q8_0, K-quants, ...; Section III-B,
weight-only quantisation "from INT8 to INT4").  The paper names the schemes but
does not define them; the definitions taken here are the published GGUF (ggml)
block formats, for the three basic 32-element blocks:

  Q4_0  18 bytes: f16 d, then 16 bytes qs.   W = (q - 8) * d
  Q4_1  20 bytes: f16 d, f16 m, then qs.     W = q * d + m
  Q8_0  34 bytes: f16 d, then 32 int8 qs.    W = q * d

with, for the 4-bit blocks, element j (0 <= j < 16) in the low nibble of qs[j]
and element j + 16 in its high nibble.  A tensor row of K weights is K / 32
consecutive blocks; rows are consecutive.  f16 values are little-endian IEEE
binary16.

Also here: the two internal layouts these blocks map onto exactly (beside the
int8 per-channel and int4 zero-point ones of ``oracle.quant``):

  int8 group:   int8 codes [N, K], f16 scales [N, K/32]:  W = q * s[n, k/32]
  int4 min:     packed int4 codes as in oracle.quant (k = 2j low nibble),
                f16 scales and mins [N, K/32]:              W = q * s + m

All values are computed in float64; every one is exact there.
"""
from __future__ import annotations

import numpy as np

from .quant import unpack_int4

QK = 32
BLOCK_BYTES = {"q4_0": 18, "q4_1": 20, "q8_0": 34}
# ggml tensor type ids of the three formats
TYPE_ID = {"q4_0": 2, "q4_1": 3, "q8_0": 8}


def _f16(lo, hi):
    b = (np.asarray(lo, dtype=np.uint16) | (np.asarray(hi, dtype=np.uint16) << 8)).astype(np.uint16)
    return b.view(np.float16).astype(np.float64)


def parse(blocks, fmt: str, K: int):
    """Rows of blocks [N, K/32 * bytes] -> (codes [N, K], d [N, K/32], m [N, K/32] or None).

    4-bit codes are the unsigned nibbles 0..15 in element order; 8-bit codes
    are signed."""
    b = np.asarray(blocks, dtype=np.uint8)
    nb = K // QK
    B = BLOCK_BYTES[fmt]
    assert K % QK == 0 and b.shape[1] == nb * B, (b.shape, K, fmt)
    blk = b.reshape(b.shape[0], nb, B)
    d = _f16(blk[:, :, 0], blk[:, :, 1])
    m = None
    if fmt == "q8_0":
        codes = blk[:, :, 2:].view(np.int8).reshape(b.shape[0], K)
        return codes, d, m
    off = 2
    if fmt == "q4_1":
        m = _f16(blk[:, :, 2], blk[:, :, 3])
        off = 4
    qs = blk[:, :, off:off + 16]
    codes = np.concatenate([qs & 0x0F, qs >> 4], axis=2)  # elements 0..15, then 16..31
    return codes.reshape(b.shape[0], K), d, m


def dequant(blocks, fmt: str, K: int):
    """Rows of blocks -> float64 weights [N, K]."""
    codes, d, m = parse(blocks, fmt, K)
    q = codes.astype(np.float64)
    g = np.arange(K) // QK
    if fmt == "q4_0":
        return (q - 8.0) * d[:, g]
    if fmt == "q4_1":
        return q * d[:, g] + m[:, g]
    return q * d[:, g]


def dequant_int8_group(q, scales):
    """Internal int8 group layout: W = q * s[n, k/32]."""
    q = np.asarray(q, dtype=np.int8).astype(np.float64)
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    assert s.shape == (q.shape[0], q.shape[1] // QK)
    return q * s[:, np.arange(q.shape[1]) // QK]


def dequant_int4_min(packed, scales, mins):
    """Internal int4 min layout: W = q * s + m per 32-k group."""
    q = unpack_int4(packed).astype(np.float64)
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    m = np.asarray(mins, dtype=np.float16).astype(np.float64)
    assert s.shape == (q.shape[0], q.shape[1] // QK) and m.shape == s.shape
    g = np.arange(q.shape[1]) // QK
    return q * s[:, g] + m[:, g]
