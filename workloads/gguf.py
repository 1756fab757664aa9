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


# --- K-quants: 256-weight super-blocks -------------------------------------

QK_K = 256
KQ_BLOCK_BYTES = {"q4_k": 144, "q6_k": 210}


def pack_q4_k(codes, d, dmin, sc, mn) -> np.ndarray:
    """codes [N, K] 0..15, d / dmin [N, K/256], sc / mn [N, K/32] in 0..63 ->
    Q4_K super-blocks [N, K/256*144]: f16 d, f16 dmin, the twelve scale bytes
    (sub-blocks 0-3: scale and min in the low six bits of bytes 0-3 / 4-7;
    sub-blocks 4-7: low four bits of scale and min in bytes 8-11, their top
    two bits in the top bits of bytes 0-3 / 4-7), then four runs of 32 bytes,
    byte l of run c holding weights 64c + l (low nibble) and 64c + 32 + l."""
    q = np.asarray(codes, dtype=np.int64)
    N, K = q.shape
    nb = K // QK_K
    out = np.zeros((N, nb, 144), dtype=np.uint8)
    out[:, :, 0:2] = np.asarray(d, dtype=np.float16).reshape(N, nb, 1).view(np.uint8)
    out[:, :, 2:4] = np.asarray(dmin, dtype=np.float16).reshape(N, nb, 1).view(np.uint8)
    s = np.asarray(sc, dtype=np.int64).reshape(N, nb, 8)
    m = np.asarray(mn, dtype=np.int64).reshape(N, nb, 8)
    out[:, :, 4:8] = (s[:, :, 0:4] | ((s[:, :, 4:8] >> 4) << 6)).astype(np.uint8)
    out[:, :, 8:12] = (m[:, :, 0:4] | ((m[:, :, 4:8] >> 4) << 6)).astype(np.uint8)
    out[:, :, 12:16] = ((s[:, :, 4:8] & 15) | ((m[:, :, 4:8] & 15) << 4)).astype(np.uint8)
    runs = q.reshape(N, nb, 4, 64)
    out[:, :, 16:144] = (runs[..., 0:32] | (runs[..., 32:64] << 4)).reshape(N, nb, 128).astype(np.uint8)
    return out.reshape(N, nb * 144)


def pack_q6_k(codes, d, sc) -> np.ndarray:
    """codes [N, K] in -32..31, d [N, K/256], sc [N, K/16] int8 -> Q6_K
    super-blocks [N, K/256*210]: ql, qh, the sixteen scales, f16 d.  With
    u = code + 32, per half h and l < 32: ql[64h + l] = low four bits of
    u[128h + l] | those of u[128h + 64 + l] << 4; ql[64h + 32 + l] likewise
    for u[128h + 32 + l] and u[128h + 96 + l]; qh[32h + l] = the top two bits
    of u[128h + l], u[128h + 32 + l], u[128h + 64 + l], u[128h + 96 + l] at
    bits 0, 2, 4, 6."""
    u = np.asarray(codes, dtype=np.int64) + 32
    N, K = u.shape
    nb = K // QK_K
    out = np.zeros((N, nb, 210), dtype=np.uint8)
    h = u.reshape(N, nb, 2, 4, 32)  # [.., half, quarter, l]
    ql = np.concatenate([(h[..., 0, :] & 15) | ((h[..., 2, :] & 15) << 4),
                         (h[..., 1, :] & 15) | ((h[..., 3, :] & 15) << 4)], axis=3)  # [.., half, 64]
    qh = (h[..., 0, :] >> 4) | ((h[..., 1, :] >> 4) << 2) | ((h[..., 2, :] >> 4) << 4) | ((h[..., 3, :] >> 4) << 6)
    out[:, :, 0:128] = ql.reshape(N, nb, 128).astype(np.uint8)
    out[:, :, 128:192] = qh.reshape(N, nb, 64).astype(np.uint8)
    out[:, :, 192:208] = np.asarray(sc, dtype=np.int8).reshape(N, nb, 16).view(np.uint8)
    out[:, :, 208:210] = np.asarray(d, dtype=np.float16).reshape(N, nb, 1).view(np.uint8)
    return out.reshape(N, nb * 210)


def random_kquant_blocks(rng, N: int, K: int, fmt: str) -> np.ndarray:
    """Every code, scale and min value with equal probability; d, dmin =
    2^U(-12, -8) * (1 + U(0,1)) stored as f16 (d negative half the time for Q6_K)."""
    nb = K // QK_K
    d = np.exp2(rng.uniform(-12, -8, size=(N, nb))) * (1 + rng.random((N, nb)))
    if fmt == "q4_k":
        dmin = np.exp2(rng.uniform(-12, -8, size=(N, nb))) * (1 + rng.random((N, nb)))
        return pack_q4_k(rng.integers(0, 16, size=(N, K)), d, dmin, rng.integers(0, 64, size=(N, K // 32)),
                         rng.integers(0, 64, size=(N, K // 32)))
    d = d * rng.choice([-1.0, 1.0], size=(N, nb))
    return pack_q6_k(rng.integers(-32, 32, size=(N, K)), d, rng.integers(-128, 128, size=(N, K // 16)))
