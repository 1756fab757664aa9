"""GPU parity of the GGUF path: rlx_gguf_repack rewrites Q4_0 / Q4_1 / Q8_0
blocks into the int4 zero-point / int4 min / int8 group layouts (and the
K-quants Q4_K / Q6_K into int4 min / int8 group-16), and
rlx_dequant_matmul multiplies with them (the tiled path for many rows, the
few-row path for 1..16), through the C ABI, against ``oracle.gguf``.

* Repack + dequantisation alone is bit-exact: every weight of these blocks is
  exact in fp32.
* The matmul is bounded by fp32 accumulation, bf16 output rounding, the bf16
  rounding of each weight on the tiled path (2^-9 of |W|), and the few-row
  path's offset arithmetic: 2^-9 sum_k |x_k| (|s| + |m|) of the block's scale
  and min (see test_gpu_gemv.py for the int4 derivation; int8 groups add
  less).
"""
import numpy as np
import pytest

import oracle
from gpu_helpers import assert_within, gemm_tolerance, to_bf16_exact
from workloads import gguf as wg

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

FMTS = ("q4_0", "q4_1", "q8_0")


@pytest.fixture(scope="module")
def rlx():
    import paper_2609_37916_amd as m
    m.lib()
    return m


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device="cuda", dtype=dtype) if dtype is not None else t.to("cuda")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("N,K", [(64, 64), (256, 384), (384, 1536)])
def test_repack_and_unpack_bit_exact(rlx, fmt, N, K):
    blocks = wg.random_blocks(np.random.default_rng(700 + N + K), N, K, fmt)
    scheme, codes, scales, zeros = rlx.gguf_repack(_dev(blocks), fmt, N=N, K=K)
    assert scheme == {"q4_0": rlx.Q_INT4_GROUP_ZP, "q4_1": rlx.Q_INT4_GROUP_MIN, "q8_0": rlx.Q_INT8_GROUP}[fmt]
    got = rlx.dequant_unpack(codes, scheme=scheme, scales=scales, zeros=zeros, N=N, K=K).cpu().numpy()
    want = oracle.gguf.dequant(blocks, fmt, K).astype(np.float32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def _case(rlx, fmt, M, N, K, epi, seed):
    rng = np.random.default_rng(seed)
    x = to_bf16_exact(rng.normal(0, 1, (M, K)))
    blocks = wg.quantize(rng.normal(0, 0.02, (N, K)).astype(np.float32), fmt)
    b = rng.normal(0, 0.5, N).astype(np.float32)
    r = to_bf16_exact(rng.normal(0, 1, (M, N)))
    scheme, codes, scales, zeros = rlx.gguf_repack(_dev(blocks), fmt, N=N, K=K)
    code = {"none": rlx.EPI_NONE, "bias": rlx.EPI_BIAS, "gelu": rlx.EPI_BIAS_GELU, "residual": rlx.EPI_BIAS_RESIDUAL}[epi]
    y = rlx.dequant_matmul(_dev(x, torch.bfloat16), codes, scheme=scheme, scales=scales, zeros=zeros, group_size=32,
                           N=N, bias=_dev(b, torch.float32), residual=_dev(r, torch.bfloat16), epi=code)
    torch.cuda.synchronize()
    w = oracle.gguf.dequant(blocks, fmt, K)
    ref = oracle.linear(x, w, None if epi == "none" else b)
    pre = ref.copy() if epi == "gelu" else None
    if epi == "gelu":
        ref = oracle.gelu(ref)
    if epi == "residual":
        ref = ref + r
    _, d, m = oracle.gguf.parse(blocks, fmt, K)
    sm = np.abs(np.repeat(d, 32, axis=1)) + (np.abs(np.repeat(m, 32, axis=1)) if m is not None else 0.0)
    tol = (gemm_tolerance(x, w, ref, out_bf16=True, weight_rel=2.0 ** -9, pre=pre) +
           2.0 ** -9 * (np.abs(x.astype(np.float64)) @ sm.T) + 2.0 ** -24 * 4 * np.abs(ref))
    return y.float().cpu().numpy(), ref, tol


# few-row shapes (1..16 rows, K % 128 == 0) and tiled ones (more rows, K % 128 != 0, or 128 KB of x;
# K >= 1024 takes the LDS-DMA kernel, with 64 x 128 tiles from N = 1024)
SHAPES = [(1, 256, 1024), (5, 1152, 384), (16, 384, 1536), (3, 128, 192), (33, 384, 1536), (300, 1536, 384),
          (16, 512, 4096), (40, 1024, 1024)]


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,N,K", SHAPES)
def test_gguf_matmul_parity(rlx, fmt, M, N, K):
    epi = ("bias", "gelu", "residual", "none")[(M + N) % 4]
    got, ref, tol = _case(rlx, fmt, M, N, K, epi, 900 + M + N + K)
    assert_within(got, ref, tol, f"gguf {fmt} {epi} {M}x{N}x{K}")


@pytest.mark.parametrize("fmt", FMTS)
def test_every_epilogue_few_rows(rlx, fmt):
    for epi in ("none", "bias", "gelu", "residual"):
        got, ref, tol = _case(rlx, fmt, 7, 256, 512, epi, 31)
        assert_within(got, ref, tol, f"gguf {fmt} {epi}")


def test_binding_rejects_a_short_block_tensor(rlx):
    blocks = _dev(wg.random_blocks(np.random.default_rng(0), 64, 64, "q4_0"))
    with pytest.raises(ValueError):
        rlx.gguf_repack(blocks, "q4_0", N=64, K=128)  # block tensor too small for the shape
    with pytest.raises(ValueError):
        rlx.gguf_repack(blocks, 6, N=64, K=64)  # Q5_0 is not supported


# --- K-quants -----------------------------------------------------------------

KFMTS = ("q4_k", "q6_k")


def _kq_internal_w(blocks, fmt, K):
    kind, c, s, m = oracle.gguf.kquant_internal(blocks, fmt, K)
    if kind == "int4_min":
        return kind, c, s, m, oracle.gguf.dequant_int4_min(c, s, m)
    return kind, c, s, m, oracle.gguf.dequant_int8_group16(c, s)


@pytest.mark.parametrize("fmt", KFMTS)
@pytest.mark.parametrize("N,K", [(64, 256), (256, 512), (384, 1536)])
def test_kquant_repack_matches_the_oracle(rlx, fmt, N, K):
    """Q4_K -> int4 with mins, Q6_K -> int8 with a scale per 16: codes,
    f16 scales and mins bit for bit as the oracle composes and rounds them;
    the unpacked weights bit for bit as the oracle's layout values, and
    within 2^-11 (|s q| + |m|) of the format's own values."""
    blocks = wg.random_kquant_blocks(np.random.default_rng(810 + N + K), N, K, fmt)
    scheme, codes, scales, zeros = rlx.gguf_repack(_dev(blocks), fmt, N=N, K=K)
    kind, c, s, m, w = _kq_internal_w(blocks, fmt, K)
    assert scheme == (rlx.Q_INT4_GROUP_MIN if fmt == "q4_k" else rlx.Q_INT8_GROUP16)
    assert np.array_equal(codes.cpu().numpy().view(np.uint8), c.view(np.uint8))
    assert np.array_equal(scales.cpu().numpy().view(np.uint16), s.view(np.uint16))
    if m is not None:
        assert np.array_equal(zeros.cpu().numpy().view(np.uint16), m.view(np.uint16))
    else:
        assert zeros is None
    got = rlx.dequant_unpack(codes, scheme=scheme, scales=scales, zeros=zeros, group_size=16 if fmt == "q6_k" else 32,
                             N=N, K=K).cpu().numpy()
    assert np.array_equal(got.view(np.uint32), w.astype(np.float32).view(np.uint32))
    gs, qmax = (32, 15) if fmt == "q4_k" else (16, 32)
    bound = 2.0 ** -11 * 1.001 * (np.repeat(np.abs(s.astype(np.float64)), gs, axis=1) * qmax +
                                  (np.repeat(np.abs(m.astype(np.float64)), gs, axis=1) if m is not None else 0.0))
    assert np.all(np.abs(got - oracle.gguf.dequant_k(blocks, fmt, K)) <= bound)


# rows 1..300: 1 and 7 rows take the few-row kernel, the others the tiled path (16 x 4096 is past the
# few-row kernel's 64 KB of activations); K >= 1024 takes the LDS-DMA kernel
KSHAPES = [(1, 256, 512), (7, 384, 512), (40, 1024, 1024), (300, 384, 1536), (16, 512, 4096)]


def _few_rows(M, K):
    return 1 <= M <= 16 and K % 128 == 0 and M * K * 2 <= 64 * 1024


def _kq_tolerance(x, w, ref, fmt, s, m, few_rows, pre=None):
    """fp32 accumulation and bf16 output (gemm_tolerance), the tiled path's
    bf16 rounding of each weight (2^-9 |W|), the scaled fp32 group sums
    (4 x 2^-24 |y|) and, for Q4_K's int4-min layout on the few-row path, the
    offset arithmetic 2^-9 sum_k |x_k| (|s| + |m|) of test_gpu_gemv.py's
    derivation."""
    tol = gemm_tolerance(x, w, ref, out_bf16=True, weight_rel=2.0 ** -9, pre=pre) + 2.0 ** -24 * 4 * np.abs(ref)
    if few_rows and m is not None:
        sm = np.repeat(np.abs(s.astype(np.float64)) + np.abs(m.astype(np.float64)), 32, axis=1)
        tol = tol + 2.0 ** -9 * (np.abs(x.astype(np.float64)) @ sm.T)
    return tol


@pytest.mark.parametrize("fmt", KFMTS)
@pytest.mark.parametrize("M,N,K", KSHAPES)
def test_kquant_matmul_parity(rlx, fmt, M, N, K):
    """Against the oracle on the repacked layout's weights (whose distance to
    the format's values is the repack test's bound): fp32 accumulation, bf16
    output rounding and the tiled path's bf16 rounding of each weight."""
    rng = np.random.default_rng(1200 + M + N + K)
    x = to_bf16_exact(rng.normal(0, 1, (M, K)))
    blocks = wg.random_kquant_blocks(rng, N, K, fmt)
    b = rng.normal(0, 0.5, N).astype(np.float32)
    epi = ("bias", "gelu", "none")[(M + K) % 3]
    scheme, codes, scales, zeros = rlx.gguf_repack(_dev(blocks), fmt, N=N, K=K)
    code = {"none": rlx.EPI_NONE, "bias": rlx.EPI_BIAS, "gelu": rlx.EPI_BIAS_GELU}[epi]
    y = rlx.dequant_matmul(_dev(x, torch.bfloat16), codes, scheme=scheme, scales=scales, zeros=zeros,
                           group_size=16 if fmt == "q6_k" else 32, N=N, bias=_dev(b, torch.float32), epi=code)
    torch.cuda.synchronize()
    _, _, s, m, w = _kq_internal_w(blocks, fmt, K)
    ref = oracle.linear(x, w, None if epi == "none" else b)
    pre = None
    if epi == "gelu":
        pre, ref = ref, oracle.gelu(ref)
    tol = _kq_tolerance(x, w, ref, fmt, s, m, _few_rows(M, K), pre=pre)
    assert_within(y.float().cpu().numpy(), ref, tol, f"gguf {fmt} {epi} {M}x{N}x{K}")


@pytest.mark.parametrize("fmt", KFMTS)
@pytest.mark.parametrize("M", [1, 8])
def test_kquant_decode_shape_sampled_columns(rlx, fmt, M):
    """The decode-sized product of the dequantising GEMV benchmark (N 14336,
    K 4096) on the few-row kernel, 96 sampled output columns against the
    oracle (which dequantises only those weight rows)."""
    N, K = 14336, 4096
    rng = np.random.default_rng(7300 + M + len(fmt))
    x = to_bf16_exact(rng.normal(0, 1, (M, K)))
    blocks = wg.random_kquant_blocks(rng, N, K, fmt)
    b = rng.normal(0, 0.5, N).astype(np.float32)
    cols = np.sort(np.concatenate([rng.choice(N, 94, replace=False), [0, N - 1]]))
    scheme, codes, scales, zeros = rlx.gguf_repack(_dev(blocks), fmt, N=N, K=K)
    y = rlx.dequant_matmul(_dev(x, torch.bfloat16), codes, scheme=scheme, scales=scales, zeros=zeros,
                           group_size=16 if fmt == "q6_k" else 32, N=N, bias=_dev(b, torch.float32), epi=rlx.EPI_BIAS)
    torch.cuda.synchronize()
    _, _, s, m, w = _kq_internal_w(blocks[cols], fmt, K)
    ref = oracle.linear(x, w, b[cols])
    tol = _kq_tolerance(x, w, ref, fmt, s, m, few_rows=True)
    assert_within(y.float().cpu().numpy()[:, cols], ref, tol, f"decode shape {fmt} M={M}")
