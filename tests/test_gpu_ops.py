"""GPU parity of the single-kernel entry points against the CPU oracle
(rlx_dequant_matmul, rlx_dequant_unpack, rlx_masked_attention), called
through the C ABI via the Python binding."""
import math

import numpy as np
import pytest

import oracle
import workloads
from gpu_helpers import BF16_REL, assert_within, gemm_tolerance, to_bf16_exact

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def rlx():
    import paper_2609_37916_amd as m
    m.lib()
    return m


def _dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


EPIS = ["none", "bias", "gelu", "residual"]


def _oracle_gemm(x, w, b, res, epi):
    y = oracle.linear(x, w, None if epi == "none" else b)
    if epi == "gelu":
        y = oracle.gelu(y)
    if epi == "residual":
        y = y + res
    return y


def _epi_code(rlx, epi):
    return {"none": rlx.EPI_NONE, "bias": rlx.EPI_BIAS, "gelu": rlx.EPI_BIAS_GELU,
            "residual": rlx.EPI_BIAS_RESIDUAL}[epi]


# (M, N, K): ragged M tails, every N/K the encoder uses, and tile-boundary cases
GEMM_SHAPES = [(1, 64, 64), (77, 384, 384), (300, 1152, 384), (257, 1536, 384), (200, 384, 1536), (4096, 384, 384),
               (513, 128, 192)]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("epi", EPIS)
@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_dense(rlx, dt, epi, M, N, K):
    rng = np.random.default_rng(1000 + M + N + K)
    x = rng.normal(0, 1, (M, K)).astype(np.float32)
    w = rng.normal(0, 0.05, (N, K)).astype(np.float32)
    b = rng.normal(0, 0.5, N).astype(np.float32)
    r = rng.normal(0, 1, (M, N)).astype(np.float32)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    if dt == "bf16":
        x, w, r = to_bf16_exact(x), to_bf16_exact(w), to_bf16_exact(r)
    y = rlx.dequant_matmul(_dev(x, tdt), _dev(w, tdt), bias=_dev(b, torch.float32), residual=_dev(r, tdt),
                           epi=_epi_code(rlx, epi))
    got = y.float().cpu().numpy()
    ref = _oracle_gemm(x, w, b, r, epi)
    pre = oracle.linear(x, w, b) if epi == "gelu" else None
    tol = gemm_tolerance(x, w, ref, out_bf16=dt == "bf16", pre=pre)
    assert_within(got, ref, tol, f"gemm {dt} {epi} {M}x{N}x{K}")


def _rne_bf16_bits(f32):
    """IEEE round-to-nearest-even of binary32 to bfloat16 bits, for finite
    values and infinities."""
    u = np.asarray(f32, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


# signed zeros, largest finite (rounds to infinity), infinities, and ties / near-ties next to 1.0
SPECIAL_F32_BITS = [0x00000000, 0x80000000, 0x7F7FFFFF, 0xFF7FFFFF, 0x7F800000, 0xFF800000, 0x3F808000, 0x3F818000,
                    0x3F807FFF, 0x3F808001, 0xBF808000, 0xBF818000]


@pytest.mark.parametrize("N", [384, 1536])
def test_bf16_output_rounding_is_round_to_nearest_even(rlx, N):
    """With x = 0 the bias epilogue's bf16 output is 0 + bias rounded once:
    checked bit for bit on random normal numbers of every exponent, low halves
    on and next to the rounding boundary (both parities of the kept bit),
    subnormals, signed zeros, overflow to infinity and infinities."""
    rng = np.random.default_rng(77 + N)
    sign = rng.integers(0, 2, N).astype(np.uint32) << np.uint32(31)
    expo = rng.integers(1, 255, N).astype(np.uint32) << np.uint32(23)
    mant = rng.integers(0, 1 << 23, N).astype(np.uint32)
    bits = sign | expo | mant
    low = np.repeat(np.array([0x8000, 0x7FFF, 0x8001, 0x0000, 0xFFFF], np.uint32), 16)
    bits[:80] = (bits[:80] & np.uint32(0xFFFF0000)) | low
    bits[80:88] = sign[80:88] | rng.integers(1, 1 << 23, 8).astype(np.uint32)  # subnormals
    bits[88:88 + len(SPECIAL_F32_BITS)] = SPECIAL_F32_BITS
    bias = bits.view(np.float32)
    M, K = 300, 64
    x = torch.zeros((M, K), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((N, K), dtype=torch.bfloat16, device="cuda")
    y = rlx.dequant_matmul(x, w, bias=_dev(bias, torch.float32), epi=rlx.EPI_BIAS)
    torch.cuda.synchronize()
    got = y.view(torch.int16).cpu().numpy().view(np.uint16)
    want = _rne_bf16_bits(np.float32(0.0) + bias)  # 0 + (-0) = +0
    bad = np.nonzero(got != want[None, :])
    assert bad[0].size == 0, (f"{bad[0].size} outputs differ; first at column {bad[1][0]}: bias bits "
                              f"{int(bits[bad[1][0]]):#010x} got {int(got[bad[0][0], bad[1][0]]):#06x} "
                              f"want {int(want[bad[1][0]]):#06x}")


@pytest.mark.parametrize("scheme", ["int8", "int4"])
@pytest.mark.parametrize("epi", EPIS)
# (K >= 1024 takes the LDS-DMA kernel: 64 x 64 tiles, or 64 x 128 from N = 1024)
@pytest.mark.parametrize("M,N,K", [(1, 64, 64), (300, 1152, 384), (129, 1536, 384), (200, 384, 1536), (100, 1024, 1024)])
def test_gemm_dequant(rlx, scheme, epi, M, N, K):
    rng = np.random.default_rng(2000 + M + N + K)
    x = to_bf16_exact(rng.normal(0, 1, (M, K)))
    wf = rng.normal(0, 0.02, (N, K)).astype(np.float32)
    b = rng.normal(0, 0.5, N).astype(np.float32)
    r = to_bf16_exact(rng.normal(0, 1, (M, N)))
    if scheme == "int8":
        q, s = workloads.quantize_int8_per_channel(wf)
        wdeq = oracle.dequant_int8(q, s)
        y = rlx.dequant_matmul(_dev(x, torch.bfloat16), _dev(q, torch.int8), scheme=rlx.Q_INT8_PER_CHANNEL,
                               scales=_dev(s, torch.float16), N=N, bias=_dev(b, torch.float32),
                               residual=_dev(r, torch.bfloat16), epi=_epi_code(rlx, epi))
        wrel = 0.0  # codes are exact in bf16; the scale multiplies the fp32 sum
    else:
        q, s, z = workloads.quantize_int4_grouped(wf, 32)
        wdeq = oracle.dequant_int4(q, s, z, 32)
        y = rlx.dequant_matmul(_dev(x, torch.bfloat16), _dev(q, torch.uint8), scheme=rlx.Q_INT4_GROUP_ZP,
                               scales=_dev(s, torch.float16), zeros=_dev(z, torch.float16), group_size=32, N=N,
                               bias=_dev(b, torch.float32), residual=_dev(r, torch.bfloat16), epi=_epi_code(rlx, epi))
        wrel = 2.0 ** -9  # each dequantised weight is rounded to bf16 before the product
    got = y.float().cpu().numpy()
    ref = _oracle_gemm(x, wdeq, b, r, epi)
    pre = oracle.linear(x, wdeq, b) if epi == "gelu" else None
    tol = gemm_tolerance(x, wdeq, ref, out_bf16=True, weight_rel=wrel, pre=pre)
    if scheme == "int8":
        tol = tol + 2.0 ** -24 * np.abs(ref) * 4  # scale applied to the fp32 sum: a few fp32 roundings
    assert_within(got, ref, tol, f"gemm {scheme} {epi} {M}x{N}x{K}")


def test_gelu_epilogue_accuracy_over_a_dense_range(rlx):
    """fp32 GEMM with an identity weight: every output is GELU(x + b) of one
    input, so the epilogue's GELU is compared directly with the erf definition
    over pre-activations densely covering [-10, 10]."""
    from gpu_helpers import GELU_REL
    M, K = 1024, 64
    x = np.linspace(-10, 10, M * K).reshape(M, K).astype(np.float32)
    w = np.eye(K, dtype=np.float32)
    b = np.zeros(K, np.float32)
    y = rlx.dequant_matmul(_dev(x, torch.float32), _dev(w, torch.float32), bias=_dev(b, torch.float32),
                           epi=rlx.EPI_BIAS_GELU)
    got = y.cpu().numpy().astype(np.float64)
    ref = oracle.gelu(x.astype(np.float64))
    assert_within(got, ref, GELU_REL * np.abs(x) + 1e-7, "GELU epilogue")


@pytest.mark.parametrize("scheme", ["int8", "int4"])
@pytest.mark.parametrize("N,K", [(64, 64), (1152, 384), (384, 1536)])
def test_dequant_unpack_bit_exact(rlx, scheme, N, K):
    rng = np.random.default_rng(3000 + N + K)
    wf = rng.normal(0, 0.02, (N, K)).astype(np.float32)
    if scheme == "int8":
        q, s = workloads.quantize_int8_per_channel(wf)
        ref = oracle.dequant_int8(q, s)
        got = rlx.dequant_unpack(_dev(q, torch.int8), scheme=rlx.Q_INT8_PER_CHANNEL, scales=_dev(s, torch.float16),
                                 N=N, K=K)
    else:
        q, s, z = workloads.quantize_int4_grouped(wf, 32)
        ref = oracle.dequant_int4(q, s, z, 32)
        got = rlx.dequant_unpack(_dev(q, torch.uint8), scheme=rlx.Q_INT4_GROUP_ZP, scales=_dev(s, torch.float16),
                                 zeros=_dev(z, torch.float16), group_size=32, N=N, K=K)
    got = got.cpu().numpy()
    assert got.dtype == np.float32
    assert np.array_equal(got.view(np.uint32), ref.astype(np.float32).view(np.uint32))


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------

KINDS = {"none": 0, "causal": 1, "sliding": 2, "custom": 3}


def _attention_case(rng, B, S, heads, lens, holes):
    H = heads * 32
    qkv = rng.normal(0, 1, (B * S, 3 * H)).astype(np.float32)
    mask = (np.arange(S)[None] < np.asarray(lens)[:, None]).astype(np.uint8)
    if holes:
        mask &= (rng.random((B, S)) < 0.7).astype(np.uint8)
    return qkv, mask


def _run_attention(rlx, qkv, mask, B, S, heads, dt, kind, window, use_mask):
    H = heads * 32
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    buf = _dev(qkv, tdt)
    out = rlx.masked_attention(buf[:, 0:H], buf[:, H:2 * H], buf[:, 2 * H:3 * H], B=B, S=S, heads=heads,
                               kind=KINDS[kind], key_mask=_dev(mask, torch.uint8) if use_mask else None,
                               window=window, row_stride=3 * H)
    return out.float().cpu().numpy().reshape(B, S, heads, 32)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("kind,window", [("custom", 0), ("none", 0), ("causal", 0), ("sliding", 1), ("sliding", 40),
                                         ("sliding", 300)])
@pytest.mark.parametrize("S", [1, 16, 77, 128, 200, 512])
def test_attention_parity(rlx, dt, kind, window, S):
    rng = np.random.default_rng(4000 + S + window + KINDS[kind])
    B, heads = 3, 4
    lens = [S, max(1, S // 3), 0 if kind == "custom" else max(1, S - 5)]
    qkv, mask = _attention_case(rng, B, S, heads, lens, holes=(kind == "custom" and S > 16))
    if dt == "bf16":
        qkv = to_bf16_exact(qkv)
    use_mask = kind == "custom" or (kind == "causal" and S > 16)
    got = _run_attention(rlx, qkv, mask, B, S, heads, dt, kind, window, use_mask)
    H = heads * 32
    q = qkv[:, :H].reshape(B, S, heads, 32)
    k = qkv[:, H:2 * H].reshape(B, S, heads, 32)
    v = qkv[:, 2 * H:].reshape(B, S, heads, 32)
    ref = oracle.masked_attention(q, k, v, KINDS[kind], mask if use_mask else None, window, 1 / math.sqrt(32))
    vmax = np.abs(v).max(axis=(1, 3), keepdims=True)  # per (b, h)
    if dt == "bf16":
        tol = BF16_REL * np.abs(ref) + 2.0 ** -7 * vmax
    else:
        tol = 1e-5 * np.abs(ref) + 1e-5 * vmax
    assert_within(got, ref, tol, f"attention {dt} {kind} w={window} S={S}")


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_attention_padding_extension_is_bit_identical(rlx, dt):
    rng = np.random.default_rng(4100)
    B, S, heads, extra = 4, 100, 12, 60
    lens = [100, 37, 64, 1]
    qkv, mask = _attention_case(rng, B, S, heads, lens, holes=False)
    if dt == "bf16":
        qkv = to_bf16_exact(qkv)
    a = _run_attention(rlx, qkv, mask, B, S, heads, dt, "custom", 0, True)
    H3 = qkv.shape[1]
    big = np.concatenate([qkv.reshape(B, S, H3), 50 * rng.normal(size=(B, extra, H3)).astype(np.float32)], axis=1)
    if dt == "bf16":
        big = to_bf16_exact(big)
    mask2 = np.concatenate([mask, np.zeros((B, extra), np.uint8)], axis=1)
    b = _run_attention(rlx, big.reshape(B * (S + extra), H3), mask2, B, S + extra, heads, dt, "custom", 0, True)
    for i, L in enumerate(lens):
        assert np.array_equal(a[i, :S], b[i, :S])


def test_attention_identical_keys_mean_of_values(rlx):
    rng = np.random.default_rng(4200)
    B, S, heads = 2, 64, 2
    H = heads * 32
    qkv = to_bf16_exact(rng.normal(0, 1, (B * S, 3 * H)))
    qkv[:, H:2 * H] = qkv[0, H:2 * H]  # every key identical
    mask = np.ones((B, S), np.uint8)
    mask[1, 40:] = 0
    got = _run_attention(rlx, qkv, mask, B, S, heads, "bf16", "custom", 0, True)
    v = qkv[:, 2 * H:].reshape(B, S, heads, 32)
    for b, L in enumerate([64, 40]):
        mean_v = v[b, :L].mean(axis=0)  # [heads, 32]
        assert_within(got[b], np.broadcast_to(mean_v, got[b].shape), BF16_REL * np.abs(mean_v) + 2.0 ** -7 *
                      np.abs(v[b, :L]).max(), "identical keys")


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("scale", [-0.3, 0.0, 2.5])
@pytest.mark.parametrize("kind,window", [("custom", 0), ("causal", 0), ("sliding", 50)])
def test_attention_scale_sign_and_zero(rlx, kind, window, scale, dt):
    """A negative scale (its sign folded into Q), a zero scale (uniform
    weights over the visible keys) and a sharp one, over several query blocks
    with a ragged sequence."""
    rng = np.random.default_rng(4300 + KINDS[kind])
    B, S, heads = 2, 300, 2
    H = heads * 32
    qkv, mask = _attention_case(rng, B, S, heads, [S, 77], holes=(kind == "custom"))
    if dt == "bf16":
        qkv = to_bf16_exact(qkv)
    use_mask = kind == "custom"
    buf = _dev(qkv, torch.bfloat16 if dt == "bf16" else torch.float32)
    got = rlx.masked_attention(buf[:, 0:H], buf[:, H:2 * H], buf[:, 2 * H:], B=B, S=S, heads=heads, kind=KINDS[kind],
                               key_mask=_dev(mask, torch.uint8) if use_mask else None, window=window, scale=scale,
                               row_stride=3 * H).float().cpu().numpy().reshape(B, S, heads, 32)
    q = qkv[:, :H].reshape(B, S, heads, 32)
    k = qkv[:, H:2 * H].reshape(B, S, heads, 32)
    v = qkv[:, 2 * H:].reshape(B, S, heads, 32)
    ref = oracle.masked_attention(q, k, v, KINDS[kind], mask if use_mask else None, window, scale)
    vmax = np.abs(v).max(axis=(1, 3), keepdims=True)
    tol = BF16_REL * np.abs(ref) + 2.0 ** -7 * vmax if dt == "bf16" else 1e-5 * np.abs(ref) + 1e-5 * vmax
    assert_within(got, ref, tol, f"attention {dt} {kind} scale={scale}")


@pytest.mark.parametrize("kind,window", [("none", 0), ("causal", 0), ("sliding", 128), ("custom", 0)])
def test_attention_benchmark_workload_full_size(rlx, kind, window):
    """The attention benchmark's own shape and launch: batch 8 x 512, 12 heads
    x 32, Q / K / V as column views of one fused [4096, 1152] bf16 buffer, key
    lengths half U[64, 512] and half 512 (the key mask for the custom kind);
    every output against the oracle."""
    rng = np.random.default_rng(11)
    B, S, heads = 8, 512, 12
    H = heads * 32
    lens = np.concatenate([rng.integers(64, S + 1, B // 2), np.full(B - B // 2, S)])
    mask = (np.arange(S)[None, :] < lens[:, None]).astype(np.uint8)
    qkv = to_bf16_exact(rng.normal(0, 1, (B * S, 3 * H)))
    use_mask = kind == "custom"
    got = _run_attention(rlx, qkv, mask, B, S, heads, "bf16", kind, window, use_mask)
    q = qkv[:, :H].reshape(B, S, heads, 32)
    k = qkv[:, H:2 * H].reshape(B, S, heads, 32)
    v = qkv[:, 2 * H:].reshape(B, S, heads, 32)
    ref = oracle.masked_attention(q, k, v, KINDS[kind], mask if use_mask else None, window, 1 / math.sqrt(32))
    tol = BF16_REL * np.abs(ref) + 2.0 ** -7 * np.abs(v).max(axis=(1, 3), keepdims=True)
    assert_within(got, ref, tol, f"attention {kind} batch 8 x 512")
