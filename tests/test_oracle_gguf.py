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
