"""Pins of the GGUF block oracle (CPU only).

Each check ties ``oracle.gguf`` to something other than itself: the block
sizes and bits per weight the formats are published with, hand-built blocks
whose values follow from the definitions, a byte-by-byte Python loop for the
element order, the quantise -> dequantise error bound of the blocks, and the
exact equivalence of each format with an internal layout that has its own,
independently written oracle (int4 zero-point, int4 min, int8 group).
"""
import numpy as np
import pytest

import oracle
import oracle.gguf as og
from workloads import gguf as wg

FMTS = ("q4_0", "q4_1", "q8_0")


def test_block_sizes_and_bits_per_weight():
    # the published sizes: 4.5, 5.0 and 8.5 bits per weight for 32-weight blocks
    assert {f: og.BLOCK_BYTES[f] * 8 / 32 for f in FMTS} == {"q4_0": 4.5, "q4_1": 5.0, "q8_0": 8.5}
    assert og.TYPE_ID == {"q4_0": 2, "q4_1": 3, "q8_0": 8}
    rng = np.random.default_rng(0)
    for f in FMTS:
        assert wg.random_blocks(rng, 3, 96, f).shape == (3, 3 * og.BLOCK_BYTES[f])


def _block(prefix, qs):
    return np.array([list(prefix) + list(qs)], dtype=np.uint8)


def test_hand_built_blocks():
    qs = [j | ((15 - j) << 4) for j in range(16)]
    one = [0x00, 0x3C]  # f16 1.0, little-endian
    # Q4_0, d = 1: low nibbles are elements 0..15, high nibbles 16..31, minus 8
    got = og.dequant(_block(one, qs), "q4_0", 32)[0]
    assert got.tolist() == [j - 8.0 for j in range(16)] + [7.0 - j for j in range(16)]
    # Q4_1, d = 0.5 (0x3800), m = -2 (0xC000)
    got = og.dequant(_block([0x00, 0x38, 0x00, 0xC0], qs), "q4_1", 32)[0]
    assert got.tolist() == [0.5 * j - 2.0 for j in range(16)] + [0.5 * (15 - j) - 2.0 for j in range(16)]
    # Q8_0, d = 0.25 (0x3400): signed bytes in element order
    codes = [-128, -127, -1, 0, 1, 2, 126, 127] * 4
    got = og.dequant(_block([0x00, 0x34], np.array(codes, dtype=np.int8).view(np.uint8)), "q8_0", 32)[0]
    assert got.tolist() == [0.25 * c for c in codes]
    # a zero scale gives zero weights (Q4_1: just the min)
    assert not og.dequant(_block([0, 0], qs), "q4_0", 32).any()
    assert og.dequant(_block([0, 0, 0x00, 0x3C], qs), "q4_1", 32).tolist() == [[1.0] * 32]


@pytest.mark.parametrize("fmt", FMTS)
def test_element_order_matches_byte_loop(fmt):
    rng = np.random.default_rng(4)
    K = 96
    b = wg.random_blocks(rng, 2, K, fmt)
    want = np.zeros((2, K))
    B = og.BLOCK_BYTES[fmt]
    for r in range(2):
        for blk in range(K // 32):
            raw = bytes(b[r, blk * B:(blk + 1) * B])
            d = float(np.frombuffer(raw[0:2], dtype=np.float16)[0])
            if fmt == "q8_0":
                for j in range(32):
                    want[r, blk * 32 + j] = int(np.frombuffer(raw[2 + j:3 + j], dtype=np.int8)[0]) * d
                continue
            m = float(np.frombuffer(raw[2:4], dtype=np.float16)[0]) if fmt == "q4_1" else 0.0
            qs = raw[4:] if fmt == "q4_1" else raw[2:]
            for j in range(16):
                lo, hi = qs[j] & 15, qs[j] >> 4
                if fmt == "q4_0":
                    want[r, blk * 32 + j], want[r, blk * 32 + 16 + j] = (lo - 8) * d, (hi - 8) * d
                else:
                    want[r, blk * 32 + j], want[r, blk * 32 + 16 + j] = lo * d + m, hi * d + m
    assert np.array_equal(og.dequant(b, fmt, K), want)


@pytest.mark.parametrize("fmt", FMTS)
def test_quantise_dequantise_error_bound(fmt):
    """Round to nearest on the block's grid: each weight is within d/2 of its
    dequantised value (plus the f16 rounding of d, at most |q| |d| 2^-11), or
    within d where Q4_0 clips the code 16 of the block's opposite extreme."""
    rng = np.random.default_rng(9)
    w = rng.normal(0, 0.02, (8, 256)).astype(np.float32)
    b = wg.quantize(w, fmt)
    got = og.dequant(b, fmt, 256)
    _, d, m = og.parse(b, fmt, 256)
    dk = np.abs(np.repeat(d, 32, axis=1))
    qmax = {"q4_0": 8, "q4_1": 15, "q8_0": 127}[fmt]
    err = np.abs(got - w.astype(np.float64))
    tol = dk * (0.5 + qmax * 2.0 ** -10) + 1e-9
    if fmt == "q4_0":
        clipped = np.abs(w / np.where(dk == 0, 1, dk)) > 7.5
        tol = np.where(clipped, dk * (1 + qmax * 2.0 ** -10), tol)
    if fmt == "q4_1":
        tol = tol + np.abs(np.repeat(m, 32, axis=1)) * 2.0 ** -11  # m rounded to f16
    assert np.all(err <= tol), float((err - tol).max())


def test_formats_equal_their_internal_layouts():
    """Q4_0 is int4 zero-point with z = 8, s = d; Q4_1 is int4 min with s = d,
    m = m; Q8_0 is int8 group with s = d (codes re-laid out two per byte with
    k = 2j in the low nibble for the 4-bit ones)."""
    rng = np.random.default_rng(12)
    K = 128
    for fmt in FMTS:
        b = wg.random_blocks(rng, 5, K, fmt)
        codes, d, m = og.parse(b, fmt, K)
        want = og.dequant(b, fmt, K)
        s16 = d.astype(np.float16)
        if fmt == "q8_0":
            got = og.dequant_int8_group(codes, s16)
        else:
            packed = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
            if fmt == "q4_0":
                got = oracle.dequant_int4(packed, s16, np.full_like(s16, 8.0), 32)
            else:
                got = og.dequant_int4_min(packed, s16, m.astype(np.float16))
        assert np.array_equal(got, want), fmt


# --- K-quants (256-weight super-blocks) --------------------------------------

KFMTS = ("q4_k", "q6_k")


def test_kquant_block_sizes_and_bits_per_weight():
    # the published sizes: 4.5 and 6.5625 bits per weight for 256-weight super-blocks
    assert {f: og.KQ_BLOCK_BYTES[f] * 8 / 256 for f in KFMTS} == {"q4_k": 4.5, "q6_k": 6.5625}
    assert og.KQ_TYPE_ID == {"q4_k": 12, "q6_k": 14}
    rng = np.random.default_rng(1)
    for f in KFMTS:
        assert wg.random_kquant_blocks(rng, 2, 512, f).shape == (2, 2 * og.KQ_BLOCK_BYTES[f])


def test_hand_built_q4_k_super_block():
    """d = 1, dmin = 0.5; scale bytes written out by hand: sub-blocks 0-3 take
    scales 1..4 / mins 5..8 from the low six bits of bytes 0-7, sub-blocks 4-7
    scales 1, 3, 5, 7 / mins 2, 4, 6, 8 from the nibbles of bytes 8-11, plus
    top bits: byte 0 = 0xC1 adds 3 << 4 to sub-block 4's scale, byte 4 = 0x85
    adds 2 << 4 to its min.  Byte l of run c: l % 16 low, 15 - l % 16 high."""
    S = [0xC1, 2, 3, 4, 0x85, 6, 7, 8, 0x21, 0x43, 0x65, 0x87]
    sc = [1, 2, 3, 4, 1 | 3 << 4, 3, 5, 7]
    mn = [5, 6, 7, 8, 2 | 2 << 4, 4, 6, 8]
    qs = [(l % 16) | ((15 - l % 16) << 4) for l in range(32)] * 4
    blk = np.array([[0x00, 0x3C, 0x00, 0x38] + S + qs], dtype=np.uint8)
    got = og.dequant_k(blk, "q4_k", 256)[0]
    want = []
    for c in range(4):
        want += [sc[2 * c] * (l % 16) - 0.5 * mn[2 * c] for l in range(32)]
        want += [sc[2 * c + 1] * (15 - l % 16) - 0.5 * mn[2 * c + 1] for l in range(32)]
    assert got.tolist() == want


def test_hand_built_q6_k_super_block():
    """d = 0.25; every ql byte 0x21 (low nibble 1, high 2), every qh byte 0xE4
    (bit pairs 0, 1, 2, 3 from the bottom): the four quarters of each half get
    the 6-bit values 1, 17, 34, 50, i.e. codes -31, -15, 2, 18; scales
    1, -1, 2, -2, ... per 16 weights."""
    scales = [(s // 2 + 1) * (1 if s % 2 == 0 else -1) for s in range(16)]
    blk = np.array([[0x21] * 128 + [0xE4] * 64 + list(np.array(scales, np.int8).view(np.uint8)) + [0x00, 0x34]],
                   dtype=np.uint8)
    got = og.dequant_k(blk, "q6_k", 256)[0]
    quarter = [-31, -15, 2, 18]
    want = [0.25 * scales[i // 16] * quarter[(i % 128) // 32] for i in range(256)]
    assert got.tolist() == want


def _q4_k_bit_address(raw, i):
    """Weight i of one Q4_K super-block, read by its bit address."""
    f16 = lambda o: float(np.frombuffer(raw[o:o + 2], dtype=np.float16)[0])
    d, dmin, S = f16(0), f16(2), raw[4:16]
    j = i // 32
    if j < 4:
        sc, mn = S[j] % 64, S[j + 4] % 64
    else:
        sc = S[j + 4] % 16 + (S[j - 4] // 64) * 16
        mn = S[j + 4] // 16 + (S[j] // 64) * 16
    c, r = divmod(i, 64)
    byte = raw[16 + 32 * c + r % 32]
    q = byte % 16 if r < 32 else byte // 16
    return d * sc * q - dmin * mn


def _q6_k_bit_address(raw, i):
    """Weight i of one Q6_K super-block, read by its bit address."""
    d = float(np.frombuffer(raw[208:210], dtype=np.float16)[0])
    sc = int(np.frombuffer(raw[192 + i // 16:193 + i // 16], dtype=np.int8)[0])
    h, r = divmod(i, 128)
    quarter, l = divmod(r, 32)
    lo_byte = raw[64 * h + l + (32 if quarter in (1, 3) else 0)]
    lo = lo_byte % 16 if quarter < 2 else lo_byte // 16
    hi = (raw[128 + 32 * h + l] >> (2 * quarter)) % 4
    return d * sc * (lo + 16 * hi - 32)


@pytest.mark.parametrize("fmt", KFMTS)
def test_kquant_element_order_matches_bit_addresses(fmt):
    rng = np.random.default_rng(5)
    K = 512
    b = wg.random_kquant_blocks(rng, 2, K, fmt)
    B = og.KQ_BLOCK_BYTES[fmt]
    read = _q4_k_bit_address if fmt == "q4_k" else _q6_k_bit_address
    want = np.array([[read(bytes(b[r, (i // 256) * B:(i // 256 + 1) * B]), i % 256) for i in range(K)]
                     for r in range(2)])
    assert np.array_equal(og.dequant_k(b, fmt, K), want)


@pytest.mark.parametrize("fmt", KFMTS)
def test_kquant_internal_layouts(fmt):
    """With d and dmin powers of two the composed scales are exact in f16 and
    the repacked layout holds the same numbers; with any d they are within
    2^-11 (|s q| + |m|) (one f16 rounding of each composed value)."""
    rng = np.random.default_rng(13)
    K, N = 512, 4
    nb = K // 256
    if fmt == "q4_k":
        codes = rng.integers(0, 16, (N, K))
        sc, mn = rng.integers(0, 64, (N, K // 32)), rng.integers(0, 64, (N, K // 32))
        exact = wg.pack_q4_k(codes, np.exp2(rng.integers(-14, -6, (N, nb))), np.exp2(rng.integers(-14, -6, (N, nb))),
                             sc, mn)
        general = wg.random_kquant_blocks(rng, N, K, fmt)
    else:
        codes = rng.integers(-32, 32, (N, K))
        exact = wg.pack_q6_k(codes, -np.exp2(rng.integers(-14, -6, (N, nb))), rng.integers(-128, 128, (N, K // 16)))
        general = wg.random_kquant_blocks(rng, N, K, fmt)

    def internal(b):
        kind, c, s, m = og.kquant_internal(b, fmt, K)
        if kind == "int4_min":
            return og.dequant_int4_min(c, s, m), s, m
        return og.dequant_int8_group16(c, s), s, None

    got, _, _ = internal(exact)
    assert np.array_equal(got, og.dequant_k(exact, fmt, K))
    got, s, m = internal(general)
    want = og.dequant_k(general, fmt, K)
    gs = 32 if fmt == "q4_k" else 16
    qmax = 15 if fmt == "q4_k" else 32
    bound = 2.0 ** -11 * 1.001 * (np.repeat(np.abs(s.astype(np.float64)), gs, axis=1) * qmax +
                          (np.repeat(np.abs(m.astype(np.float64)), gs, axis=1) if m is not None else 0.0))
    assert np.all(np.abs(got - want) <= bound)
    assert np.any(got != want)  # the rounding is real for general scales
