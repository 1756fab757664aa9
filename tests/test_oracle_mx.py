"""Pins of the block-scaled minifloat matmul oracle (CPU only).

Each check ties ``oracle.mx`` to something other than itself: values the OCP
MX v1.0 format definitions fix (largest normal, smallest subnormal, the code
of 1.0, the whole FP4 grid, the special codes), an independent library
decoder (torch's float8_e4m3fn / float8_e5m2 for all 256 codes), the grid
structure of every format, bit-by-bit unpacking of the packed layouts, and an
exact rational brute force of the matmul on small shapes.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from workloads import mx as wmx

FORMATS = ("e4m3", "e5m2", "e2m3", "e3m2", "e2m1")


def test_decode_values_fixed_by_the_format_definitions():
    d = oracle.mx.decode
    # E4M3: bias 7, 3 mantissa bits, no infinities, S.1111.111 is NaN
    assert d([0x00, 0x01, 0x07, 0x08, 0x38, 0x7E, 0xFE], "e4m3").tolist() == \
        [0.0, 2.0 ** -9, 7 * 2.0 ** -9, 2.0 ** -6, 1.0, 448.0, -448.0]
    assert np.isnan(d([0x7F, 0xFF], "e4m3")).all()
    # E5M2: bias 15, IEEE-like specials
    assert d([0x01, 0x04, 0x3C, 0x7B, 0xFB], "e5m2").tolist() == [2.0 ** -16, 2.0 ** -14, 1.0, 57344.0, -57344.0]
    assert d([0x7C, 0xFC], "e5m2").tolist() == [np.inf, -np.inf]
    assert np.isnan(d([0x7D, 0x7E, 0x7F, 0xFD, 0xFE, 0xFF], "e5m2")).all()
    # FP6
    assert d([0x01, 0x08, 0x1F, 0x3F], "e2m3").tolist() == [0.125, 1.0, 7.5, -7.5]
    assert d([0x01, 0x0C, 0x1F, 0x3F], "e3m2").tolist() == [0.0625, 1.0, 28.0, -28.0]
    # FP4: the whole grid
    assert d(np.arange(16), "e2m1").tolist() == [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0,
                                                 -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0]
    # E8M0 scales
    s = oracle.mx.decode_scale([0, 126, 127, 128, 254])
    assert s.tolist() == [2.0 ** -127, 0.5, 1.0, 2.0, 2.0 ** 127]
    assert np.isnan(oracle.mx.decode_scale([255])).all()


def test_float8_decode_matches_torch_for_every_code():
    torch = pytest.importorskip("torch")
    codes = np.arange(256, dtype=np.uint8)
    for fmt, dt in (("e4m3", torch.float8_e4m3fn), ("e5m2", torch.float8_e5m2)):
        ref = torch.from_numpy(codes.copy()).view(dt).to(torch.float64).numpy()
        got = oracle.mx.decode(codes, fmt)
        assert np.array_equal(np.isnan(ref), np.isnan(got)), fmt
        fin = ~np.isnan(ref)
        assert np.array_equal(ref[fin], got[fin]), fmt


@pytest.mark.parametrize("fmt", FORMATS)
def test_grid_structure(fmt):
    """Positive codes in order are increasing; the step from code c-1 to c is
    the spacing 2^(e - bias - mbits) of c-1's binade e (subnormals share the
    first normal binade's spacing), and every negative code mirrors its
    positive code."""
    ebits, mbits, bias = oracle.mx.MX_FORMATS[fmt]
    nbits = 1 + ebits + mbits
    pos = np.arange(1 << (nbits - 1))
    v = oracle.mx.decode(pos, fmt)
    fin = np.isfinite(v)
    vf = v[fin]
    assert np.all(np.diff(vf) > 0)
    for c in pos[fin][1:]:
        e = max((int(c) - 1) >> mbits, 1)
        assert v[c] - v[c - 1] == 2.0 ** (e - bias - mbits), (fmt, c)
    neg = oracle.mx.decode(pos | (1 << (nbits - 1)), fmt)
    assert np.array_equal(neg[fin], -v[fin])


def _bit_loop_unpack(packed, bits, K):
    out = np.zeros((packed.shape[0], K), dtype=np.uint8)
    for r in range(packed.shape[0]):
        stream = []
        for byte in packed[r]:
            stream += [(int(byte) >> i) & 1 for i in range(8)]
        for k in range(K):
            out[r, k] = sum(stream[k * bits + i] << i for i in range(bits))
    return out


@pytest.mark.parametrize("fmt", FORMATS)
def test_unpack_matches_bit_loop(fmt):
    rng = np.random.default_rng(3)
    K = 64
    bits = oracle.mx.code_bits(fmt)
    packed = rng.integers(0, 256, size=(3, K * bits // 8), dtype=np.uint8)
    assert np.array_equal(oracle.mx.unpack(packed, fmt, K), _bit_loop_unpack(packed, bits, K))


def _frac(v):
    return Fraction(float(v))


@pytest.mark.parametrize("fa,fb", [("e4m3", "e4m3"), ("e5m2", "e2m1"), ("e2m3", "e3m2"), ("e2m1", "e2m1")])
def test_scaled_matmul_matches_exact_rational_brute_force(fa, fb):
    M, N, K = 3, 4, 64
    a, b = wmx.matmul_inputs(11, M, N, K, fa, fb)
    got = oracle.mx.scaled_matmul(a.packed, a.scales, fa, b.packed, b.scales, fb, K)
    va = oracle.mx.decode(a.codes, fa)
    vb = oracle.mx.decode(b.codes, fb)
    for m in range(M):
        for n in range(N):
            acc = Fraction(0)
            for k in range(K):
                sa = Fraction(2) ** (int(a.scales[m, k // 32]) - 127)
                sb = Fraction(2) ** (int(b.scales[n, k // 32]) - 127)
                acc += _frac(va[m, k]) * sa * _frac(vb[n, k]) * sb
            assert Fraction(float(got[m, n])) == acc, (m, n)


def test_block_scale_multiplies_its_block_only():
    fa = fb = "e4m3"
    K = 64
    a, b = wmx.matmul_inputs(5, 2, 2, K, fa, fb)
    base = oracle.mx.scaled_matmul(a.packed, a.scales, fa, b.packed, b.scales, fb, K)
    s2 = a.scales.copy()
    s2[:, 1] += 1  # second block of every A row doubled
    got = oracle.mx.scaled_matmul(a.packed, s2, fa, b.packed, b.scales, fb, K)
    A = oracle.mx.dequant(a.packed, a.scales, fa, K)
    B = oracle.mx.dequant(b.packed, b.scales, fb, K)
    second = A[:, 32:] @ B[:, 32:].T
    assert np.array_equal(got, base + second)


def test_exact_inputs_keep_float32_sums_exact():
    """The bit-exact GPU comparisons rely on these inputs: every product is a
    multiple of g = 2^-(da + db + 2) (da, db: the largest binary denominator of
    the codes' values; the two scales contribute at most 2^-2) and every
    partial sum of a 512-long dot product stays below 2^24 g, so float32 adds
    them without rounding in any order."""
    def denom_exp(v):
        return max(Fraction(float(x)).denominator.bit_length() - 1 for x in v)
    for fa, fb in [("e4m3", "e4m3"), ("e5m2", "e5m2"), ("e2m3", "e3m2"), ("e2m1", "e2m1"), ("e4m3", "e2m1")]:
        va = oracle.mx.decode(wmx.exact_codes(fa), fa)
        vb = oracle.mx.decode(wmx.exact_codes(fb), fb)
        g = 2.0 ** -(denom_exp(va) + denom_exp(vb) + 2)
        P = np.abs(va).max() * np.abs(vb).max() * 4.0
        assert 512 * P / g < 2.0 ** 24, (fa, fb)
