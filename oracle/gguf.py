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

K-quants (256-weight super-blocks, the published GGUF layouts):

  Q4_K  144 bytes: f16 d, f16 dmin, 12 bytes of 6-bit sub-block scales and
        mins, 128 bytes of nibbles.  Eight sub-blocks of 32 weights; sub-block
        j has an unsigned 6-bit scale sc_j and min mn_j:
          j < 4:  sc_j = S[j] & 63,                    mn_j = S[j+4] & 63
          j >= 4: sc_j = (S[j+4] & 15) | (S[j-4] >> 6) << 4,
                  mn_j = (S[j+4] >> 4) | (S[j] >> 6) << 4
        (S the 12 scale bytes).  The weights come in four runs of 64: byte
        32c + l holds weight 64c + l in its low nibble and 64c + 32 + l in its
        high nibble.   W = d * sc_j * q - dmin * mn_j
  Q6_K  210 bytes: 128 bytes ql (low four bits), 64 bytes qh (high two bits),
        16 int8 sub-block scales, f16 d.  Sixteen sub-blocks of 16 weights
        (weight i uses scale i / 16).  Per half h of 128 weights, with
        L = ql[64h ..], Hb = qh[32h ..] and l < 32: weight 128h + l takes
        the low nibble of L[l] and bits 0-1 of Hb[l]; 128h + 32 + l the low
        nibble of L[32 + l] and bits 2-3; 128h + 64 + l the high nibble of
        L[l] and bits 4-5; 128h + 96 + l the high nibble of L[32 + l] and bits
        6-7 (the two bits above the four).   W = d * sc_i * (q - 32)

and one more internal layout, for Q6_K's 16-weight sub-blocks:

  int8 group16: int8 codes [N, K], f16 scales [N, K/16]:   W = q * s[n, k/16]

The K-quants' composed scales d * sc_j (and dmin * mn_j, d * sc_i) carry up
to 17 (Q4_K) or 19 (Q6_K) significant bits; the internal layouts hold f16
scales, so the repack rounds them once to f16 (round to nearest even) and
the repacked weights are within 2^-11 of |s q| + |m| of the format's
values (``kquant_internal``).

All values are computed in float64; every one is exact there.
"""
from __future__ import annotations

import numpy as np

from .quant import unpack_int4

QK = 32
QK_K = 256
BLOCK_BYTES = {"q4_0": 18, "q4_1": 20, "q8_0": 34}
# ggml tensor type ids of the three formats
TYPE_ID = {"q4_0": 2, "q4_1": 3, "q8_0": 8}
KQ_BLOCK_BYTES = {"q4_k": 144, "q6_k": 210}
KQ_TYPE_ID = {"q4_k": 12, "q6_k": 14}


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


def _kq_blocks(blocks, fmt: str, K: int):
    b = np.asarray(blocks, dtype=np.uint8)
    B = KQ_BLOCK_BYTES[fmt]
    assert K % QK_K == 0 and b.shape[1] == K // QK_K * B, (b.shape, K, fmt)
    return b.reshape(b.shape[0], K // QK_K, B)


def parse_q4_k(blocks, K: int):
    """Rows of Q4_K super-blocks -> (codes [N, K] 0..15 in weight order,
    d [N, K/256], dmin [N, K/256], sc [N, K/32], mn [N, K/32])."""
    blk = _kq_blocks(blocks, "q4_k", K)
    N, nb = blk.shape[:2]
    d = _f16(blk[:, :, 0], blk[:, :, 1])
    dmin = _f16(blk[:, :, 2], blk[:, :, 3])
    S = blk[:, :, 4:16].astype(np.int64)
    sc = np.zeros((N, nb, 8), np.int64)
    mn = np.zeros((N, nb, 8), np.int64)
    sc[:, :, 0:4] = S[:, :, 0:4] & 63
    mn[:, :, 0:4] = S[:, :, 4:8] & 63
    sc[:, :, 4:8] = (S[:, :, 8:12] & 15) | ((S[:, :, 0:4] >> 6) << 4)
    mn[:, :, 4:8] = (S[:, :, 8:12] >> 4) | ((S[:, :, 4:8] >> 6) << 4)
    qs = blk[:, :, 16:144].reshape(N, nb, 4, 32)
    codes = np.concatenate([qs & 0x0F, qs >> 4], axis=3)  # run c: weights 64c .. 64c+31, then +32 .. +63
    return codes.reshape(N, K), d, dmin, sc.reshape(N, nb * 8), mn.reshape(N, nb * 8)


def parse_q6_k(blocks, K: int):
    """Rows of Q6_K super-blocks -> (codes [N, K] -32..31 in weight order,
    d [N, K/256], sc [N, K/16] signed)."""
    blk = _kq_blocks(blocks, "q6_k", K)
    N, nb = blk.shape[:2]
    ql = blk[:, :, 0:128].reshape(N, nb, 2, 64).astype(np.int64)
    qh = blk[:, :, 128:192].reshape(N, nb, 2, 32).astype(np.int64)
    sc = blk[:, :, 192:208].view(np.int8).astype(np.int64)
    d = _f16(blk[:, :, 208], blk[:, :, 209])
    lo0, lo1 = ql[..., 0:32], ql[..., 32:64]
    q = np.concatenate([
        (lo0 & 15) | (((qh >> 0) & 3) << 4),
        (lo1 & 15) | (((qh >> 2) & 3) << 4),
        (lo0 >> 4) | (((qh >> 4) & 3) << 4),
        (lo1 >> 4) | (((qh >> 6) & 3) << 4),
    ], axis=3)  # [N, nb, half, 128]
    return (q - 32).reshape(N, K), d, sc.reshape(N, nb * 16)


def dequant_k(blocks, fmt: str, K: int):
    """Rows of K-quant super-blocks -> float64 weights [N, K] (exact)."""
    if fmt == "q4_k":
        codes, d, dmin, sc, mn = parse_q4_k(blocks, K)
        sb, g = np.arange(K) // QK_K, np.arange(K) // 32
        return d[:, sb] * sc[:, g] * codes - dmin[:, sb] * mn[:, g]
    codes, d, sc = parse_q6_k(blocks, K)
    sb, g = np.arange(K) // QK_K, np.arange(K) // 16
    return d[:, sb] * sc[:, g] * codes


def dequant_int8_group16(q, scales):
    """Internal int8 group16 layout: W = q * s[n, k/16]."""
    q = np.asarray(q, dtype=np.int8).astype(np.float64)
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    assert s.shape == (q.shape[0], q.shape[1] // 16)
    return q * s[:, np.arange(q.shape[1]) // 16]


def kquant_internal(blocks, fmt: str, K: int):
    """The internal layout a K-quant tensor is repacked into, as arrays:
    Q4_K -> ("int4_min", packed codes [N, K/2] (k = 2j low nibble), f16
    scales d * sc_j, f16 mins 0 - dmin * mn_j (a zero min is +0), each [N, K/32]);
    Q6_K -> ("int8_group16", int8 codes [N, K], f16 scales d * sc_i [N, K/16], None).
    The composed scales are rounded once to f16 (nearest even)."""
    if fmt == "q4_k":
        codes, d, dmin, sc, mn = parse_q4_k(blocks, K)
        sb = np.arange(K // 32) // 8
        s = (d[:, sb] * sc).astype(np.float16)
        m = (0.0 - dmin[:, sb] * mn).astype(np.float16)  # 0 - x: a zero min is +0
        packed = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
        return "int4_min", packed, s, m
    codes, d, sc = parse_q6_k(blocks, K)
    s = (d[:, np.arange(K // 16) // 16] * sc).astype(np.float16)
    return "int8_group16", codes.astype(np.int8), s, None
