"""Seeded GGUF weight blocks (Q4_0, Q4_1, Q8_0) for the dequantising matmul.

Two generators: ``quantize`` turns float weights into blocks the way the
GGUF reference quantisers do (a block's scale from its extreme value, codes
rounded to nearest), and ``random_blocks`` draws every code value and random
finite f16 scales / mins directly.  Both only lay codes and f16 values out in
the block format (f16 d [, f16 m], then the codes; for 4-bit blocks element
j < 16 in the low nibble of byte j and element j + 16 in its high nibble);
none of the matmul's arithmetic is here.
"""
from __future__ import annotations

import numpy as np

QK = 32
BLOCK_BYTES = {"q4_0": 18, "q4_1": 20, "q8_0": 34}


def pack_blocks(codes, d, m, fmt: str) -> np.ndarray:
    """codes [N, K] (4-bit: 0..15 in element order; 8-bit: int8), d / m [N, K/32] -> blocks [N, K/32*bytes]."""
    q = np.asarray(codes)
    N, K = q.shape
    nb = K // QK
    B = BLOCK_BYTES[fmt]
    out = np.zeros((N, nb, B), dtype=np.uint8)
    out[:, :, 0:2] = np.asarray(d, dtype=np.float16).reshape(N, nb, 1).view(np.uint8)
    if fmt == "q8_0":
        out[:, :, 2:] = q.astype(np.int8).reshape(N, nb, QK).view(np.uint8)
        return out.reshape(N, nb * B)
    off = 2
    if fmt == "q4_1":
        out[:, :, 2:4] = np.asarray(m, dtype=np.float16).reshape(N, nb, 1).view(np.uint8)
        off = 4
    c = q.astype(np.uint8).reshape(N, nb, QK)
    out[:, :, off:off + 16] = (c[:, :, :16] | (c[:, :, 16:] << 4)).astype(np.uint8)
    return out.reshape(N, nb * B)


def quantize(w: np.ndarray, fmt: str) -> np.ndarray:
    """float weights [N, K] -> blocks.  Q4_0: d = x_ext / -8 with x_ext the
    block's value of largest magnitude, q = min(15, floor(x / d + 8.5));
    Q4_1: d = (max - min) / 15, m = min, q = min(15, floor((x - min) / d + 0.5));
    Q8_0: d = max|x| / 127, q = round(x / d).  Codes use the unrounded d (in
    float32); d and m are stored as f16."""
    x = np.asarray(w, dtype=np.float32)
    N, K = x.shape
    blk = x.reshape(N, K // QK, QK)
    if fmt == "q4_0":
        idx = np.abs(blk).argmax(axis=2)
        ext = np.take_along_axis(blk, idx[:, :, None], axis=2)[:, :, 0]
        d = ext / np.float32(-8.0)
        inv = np.where(d != 0, np.float32(1.0) / np.where(d != 0, d, 1), 0).astype(np.float32)
        q = np.minimum(15, np.floor(blk * inv[:, :, None] + np.float32(8.5))).astype(np.int64)
        q = np.clip(q, 0, 15)
        return pack_blocks(q.reshape(N, K), d, None, fmt)
    if fmt == "q4_1":
        lo, hi = blk.min(axis=2), blk.max(axis=2)
        d = (hi - lo) / np.float32(15.0)
        inv = np.where(d != 0, np.float32(1.0) / np.where(d != 0, d, 1), 0).astype(np.float32)
        q = np.minimum(15, np.floor((blk - lo[:, :, None]) * inv[:, :, None] + np.float32(0.5))).astype(np.int64)
        q = np.clip(q, 0, 15)
        return pack_blocks(q.reshape(N, K), d, lo, fmt)
    amax = np.abs(blk).max(axis=2)
    d = amax / np.float32(127.0)
    inv = np.where(d != 0, np.float32(1.0) / np.where(d != 0, d, 1), 0).astype(np.float32)
    q = np.clip(np.rint(blk * inv[:, :, None]), -127, 127).astype(np.int64)
    return pack_blocks(q.reshape(N, K), d, None, fmt)


def random_blocks(rng, N: int, K: int, fmt: str) -> np.ndarray:
    """Every code value with equal probability; d = +-2^U(-8, -4) * (1 + U(0,1)),
    m = N(0, 0.05), both stored as f16."""
    nb = K // QK
    if fmt == "q8_0":
        codes = rng.integers(-128, 128, size=(N, K))
    else:
        codes = rng.integers(0, 16, size=(N, K))
    d = (rng.choice([-1.0, 1.0], size=(N, nb)) * np.exp2(rng.uniform(-8, -4, size=(N, nb))) *
         (1 + rng.random((N, nb))))
    m = rng.normal(0, 0.05, size=(N, nb)) if fmt == "q4_1" else None
    return pack_blocks(codes, d, m, fmt)
