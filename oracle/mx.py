"""Block-scaled minifloat matmul (test infrastructure; see package docstring).

The paper's ScaledMatMul path (Section VI, quantized inference; Section
III-B, numeric precision) multiplies matrices stored as block-scaled
minifloats -- the FP8 / FP6 / FP4 grids -- and is checked bit for bit against
an F32 reference.  The paper names the formats but does not define them; the
definitions taken here are those of the OCP Microscaling (MX) formats, v1.0:

* a block of 32 consecutive elements along K shares one scale X;
* X is E8M0: an unsigned 8-bit biased exponent, X = 2^(e - 127); e = 255 is NaN;
* element formats (sign, exponent bits, mantissa bits, exponent bias):

    E4M3  (FP8)  1, 4, 3, bias 7   no infinities; S.1111.111 is NaN; max 448
    E5M2  (FP8)  1, 5, 2, bias 15  IEEE-like: exponent 31 is Inf (m = 0) or NaN
    E2M3  (FP6)  1, 2, 3, bias 1   no Inf / NaN; max 7.5
    E3M2  (FP6)  1, 3, 2, bias 3   no Inf / NaN; max 28
    E2M1  (FP4)  1, 2, 1, bias 1   no Inf / NaN; max 6

  exponent field 0 is subnormal: (-1)^s 2^(1 - bias) (m / 2^mbits); otherwise
  (-1)^s 2^(e - bias) (1 + m / 2^mbits).
* value of element k of a row = X[k // 32] * decode(code[k]).

Storage readings (the library's layout, the same on both sides): rows are
row-major along K; FP8 codes take one byte each; FP4 codes two per byte, the
lower k in the low nibble; FP6 codes four per three bytes as a little-endian
bit stream (code i of a row occupies bits 6i .. 6i+5 of the row's bytes read
as one little-endian integer).  Scales are one byte per (row, block), [rows, K/32].

ScaledMatMul:  Y[m, n] = sum_k A(m, k) * B(n, k)  (B in the nn.Linear
convention, one row per output column), computed here in float64 on the
decoded values.  Every product of two decoded elements and two scales is a
power-of-two multiple of a small integer, so the float64 sum is exact for
every input the tests use, and equals any exactly rounded float32 result
whenever the float32 partial sums are exact.
"""
from __future__ import annotations

import numpy as np

MX_BLOCK = 32

# format name -> (exponent bits, mantissa bits, bias)
MX_FORMATS = {
    "e4m3": (4, 3, 7),
    "e5m2": (5, 2, 15),
    "e2m3": (2, 3, 1),
    "e3m2": (3, 2, 3),
    "e2m1": (2, 1, 1),
}


def code_bits(fmt: str) -> int:
    e, m, _ = MX_FORMATS[fmt]
    return 1 + e + m


def is_special(codes, fmt: str):
    """True where a code is NaN or Inf in its format."""
    c = np.asarray(codes, dtype=np.int64)
    ebits, mbits, _ = MX_FORMATS[fmt]
    mag = c & ((1 << (ebits + mbits)) - 1)
    if fmt == "e4m3":
        return mag == (1 << (ebits + mbits)) - 1          # S.1111.111
    if fmt == "e5m2":
        return (mag >> mbits) == (1 << ebits) - 1          # exponent all ones
    return np.zeros(c.shape, dtype=bool)


def decode(codes, fmt: str):
    """Element codes -> float64 values (NaN / +-Inf where the format has them)."""
    c = np.asarray(codes, dtype=np.int64)
    ebits, mbits, bias = MX_FORMATS[fmt]
    sign = np.where((c >> (ebits + mbits)) & 1, -1.0, 1.0)
    e = (c >> mbits) & ((1 << ebits) - 1)
    m = (c & ((1 << mbits) - 1)).astype(np.float64)
    frac = m / float(1 << mbits)
    val = np.where(e == 0, np.ldexp(frac, 1 - bias), np.ldexp(1.0 + frac, e - bias))
    val = sign * val
    if fmt == "e4m3":
        val = np.where(is_special(c, fmt), np.nan, val)
    elif fmt == "e5m2":
        val = np.where(is_special(c, fmt), np.where(m == 0, sign * np.inf, np.nan), val)
    return val


def decode_scale(s):
    """E8M0 scale bytes -> float64 2^(e - 127); 255 is NaN."""
    e = np.asarray(s, dtype=np.int64)
    return np.where(e == 255, np.nan, np.ldexp(1.0, e - 127))


def row_bytes(fmt: str, K: int) -> int:
    """Bytes of one stored row of K codes."""
    assert K % MX_BLOCK == 0
    return K * code_bits(fmt) // 8


def unpack(packed, fmt: str, K: int):
    """Stored rows [R, row_bytes] -> codes [R, K] (uint8)."""
    p = np.asarray(packed, dtype=np.uint8)
    R = p.shape[0]
    bits = code_bits(fmt)
    if bits == 8:
        assert p.shape == (R, K)
        return p.copy()
    if bits == 4:
        assert p.shape == (R, K // 2)
        q = np.empty((R, K), dtype=np.uint8)
        q[:, 0::2] = p & 0x0F
        q[:, 1::2] = p >> 4
        return q
    assert bits == 6 and p.shape == (R, K * 6 // 8)
    # every 3 bytes hold 4 codes: a 24-bit little-endian word, code i at bits 6i
    w = p.reshape(R, K // 4, 3).astype(np.uint32)
    word = w[:, :, 0] | (w[:, :, 1] << 8) | (w[:, :, 2] << 16)
    q = np.stack([(word >> (6 * i)) & 0x3F for i in range(4)], axis=-1)
    return q.reshape(R, K).astype(np.uint8)


def dequant(packed, scales, fmt: str, K: int):
    """Stored rows and their block scales -> float64 [R, K]."""
    v = decode(unpack(packed, fmt, K), fmt)
    x = decode_scale(scales)
    assert x.shape == (v.shape[0], K // MX_BLOCK)
    return v * np.repeat(x, MX_BLOCK, axis=1)


def scaled_matmul(a, a_scales, fa: str, b, b_scales, fb: str, K: int):
    """Y[m, n] = sum_k A(m, k) B(n, k), float64."""
    A = dequant(a, a_scales, fa, K)
    B = dequant(b, b_scales, fb, K)
    return A @ B.T
