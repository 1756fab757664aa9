"""GPU parity of every tile path rlx_dequant_matmul dispatches to, through the
C ABI, against the CPU oracle.

1. Unpacking, bit for bit, inside the product itself.  With one-hot activation
   rows (x[m, k] = 1 for k = k(m), else 0) and no epilogue, every output is one
   dequantised weight taken through the GEMM's own conversion and matrix-core
   product: y[m, n] = W[n, k(m)] plus exact zeros.  Each path's arithmetic
   makes that exact, so the bf16 output must equal round-to-nearest-even of
   the oracle's dequantised weight bit for bit:
     - int8 per channel: the code enters the matrix cores exactly and the
       epilogue multiplies by the scale, q * s, exact in fp32;
     - tiled int4 (zero-point), int8 group: (q - z) * s and q * s are exact in
       fp32 and rounded once to bf16 before the product; 1.0 times a bf16 value
       adds exactly;
     - tiled int4 min: q * s + m rounded once to fp32 (one fused multiply-add),
       then to bf16;
     - few-row int4 (integer zero-points): s (128 + q) and s (128 + z) are exact
       in fp32 and so is their difference s (q - z).
   The few-row int4-min form adds s (128 + q) and the fp32-rounded offset
   m - 128 s, two roundings instead of one: there the output may differ from
   the oracle's by one bf16 unit in the last place.
   Shapes are chosen so the dispatch takes each path: the register-staged
   kernel's 64 x 64, 64 x 128 and 128 x 128 tiles (K = 384), the LDS-DMA kernel's
   64 x 64 and 64 x 128 tiles (K >= 1024), and the few-row kernel (M <= 16).
2. Element-wise products with every epilogue at the full-size shapes that
   select the quantised 128 x 128 tile (M = 4096, N in {1152, 1536}, K = 384)
   and the dense bf16 128 x 128 tile (M = 16384), with the derived tolerances
   of the other GEMM tests.
3. The f32 output (y_dt = RLX_F32 with bf16 activations): one-hot rows give the
   exact dequantised weight wherever no weight is rounded, and element-wise
   products with an f32 residual match the oracle.
"""
import numpy as np
import pytest

import oracle
import workloads
from gpu_helpers import assert_within, gemm_tolerance, to_bf16_exact
from oracle.gguf import dequant_int4_min, dequant_int8_group

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SCHEMES = ["int8", "int4", "int8g", "int4m", "int8g16"]
EPIS = ["none", "bias", "gelu", "residual"]

# path -> (M, N, K): the dispatch rule that selects it is stated beside each
PATHS = {
    "reg64x64": (448, 384, 384),      # K < 1024, too few 64 x 128 tiles for 256 CUs
    "reg64x128": (2048, 1152, 384),   # 32 x 9 64 x 128 tiles >= 256, 16 x 9 128 x 128 tiles < 256
    "reg128x128": (4096, 1152, 384),  # 32 x 9 128 x 128 tiles >= 256
    "dma64x64": (1100, 384, 1024),    # K >= 1024, N < 1024
    "dma64x128": (1100, 1024, 1024),  # K >= 1024, N >= 1024
    "gemv": (16, 384, 1024),          # 1 <= M <= 16, K % 128 == 0, M K 2 <= 64 KB
}


@pytest.fixture(scope="module")
def rlx():
    import paper_2609_37916_amd as m
    m.lib()
    return m


def _dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def _epi_code(rlx, epi):
    return {"none": rlx.EPI_NONE, "bias": rlx.EPI_BIAS, "gelu": rlx.EPI_BIAS_GELU,
            "residual": rlx.EPI_BIAS_RESIDUAL}[epi]


def _rne_bf16_bits(f32):
    u = np.asarray(f32, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


class Weights:
    """Seeded quantised weights of one scheme and their exact dequantised
    values from the oracle (float64; the int4-min form rounded once to fp32,
    as its definition in the kernels states)."""

    def __init__(self, scheme, N, K, seed):
        rng = np.random.default_rng(seed)
        self.scheme = scheme
        wf = rng.normal(0, 0.02, (N, K)).astype(np.float32)
        self.zeros = None
        if scheme == "int8":
            self.q, self.scales = workloads.quantize_int8_per_channel(wf)
            self.w = oracle.dequant_int8(self.q, self.scales)
        elif scheme == "int4":
            self.q, self.scales, self.zeros = workloads.quantize_int4_grouped(wf, 32)
            self.w = oracle.dequant_int4(self.q, self.scales, self.zeros, 32)
        elif scheme == "int8g":
            self.q = rng.integers(-127, 128, (N, K)).astype(np.int8)
            self.scales = (rng.uniform(0.5, 2.0, (N, K // 32)) * 2e-4).astype(np.float16)
            self.w = dequant_int8_group(self.q, self.scales)
        elif scheme == "int8g16":  # GGUF Q6_K's layout: a scale per 16 weights
            self.q = rng.integers(-32, 32, (N, K)).astype(np.int8)
            self.scales = (rng.choice([-1.0, 1.0], (N, K // 16)) * rng.uniform(0.5, 2.0, (N, K // 16)) *
                           5e-4).astype(np.float16)
            self.w = oracle.gguf.dequant_int8_group16(self.q, self.scales)
        else:
            codes = rng.integers(0, 16, (N, K)).astype(np.uint8)
            self.q = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
            self.scales = (rng.uniform(0.5, 2.0, (N, K // 32)) * 3e-3).astype(np.float16)
            self.zeros = (-rng.uniform(0.0, 0.05, (N, K // 32))).astype(np.float16)  # the mins m
            self.w = dequant_int4_min(self.q, self.scales, self.zeros).astype(np.float32).astype(np.float64)

    def run(self, rlx, x, *, bias=None, residual=None, epi="none", out_dtype=None):
        scheme = {"int8": rlx.Q_INT8_PER_CHANNEL, "int4": rlx.Q_INT4_GROUP_ZP, "int8g": rlx.Q_INT8_GROUP,
                  "int4m": rlx.Q_INT4_GROUP_MIN, "int8g16": rlx.Q_INT8_GROUP16}[self.scheme]
        qd = _dev(self.q, torch.int8 if self.scheme in ("int8", "int8g", "int8g16") else torch.uint8)
        rdt = torch.float32 if out_dtype == torch.float32 else torch.bfloat16
        y = rlx.dequant_matmul(_dev(x, torch.bfloat16), qd, scheme=scheme, scales=_dev(self.scales, torch.float16),
                               zeros=None if self.zeros is None else _dev(self.zeros, torch.float16),
                               group_size=16 if self.scheme == "int8g16" else 32,
                               N=self.w.shape[0], bias=None if bias is None else _dev(bias, torch.float32),
                               residual=None if residual is None else _dev(residual, rdt), epi=_epi_code(rlx, epi),
                               out_dtype=out_dtype)
        torch.cuda.synchronize()
        return y


def _one_hot_rows(M, K, offset):
    """x[m, (m + offset) mod K] = 1: row m selects weight column k(m)."""
    k = (np.arange(M) + offset) % K
    x = np.zeros((M, K), np.float32)
    x[np.arange(M), k] = 1.0
    return x, k


@pytest.mark.parametrize("scheme", SCHEMES)
@pytest.mark.parametrize("path", sorted(PATHS))
def test_one_hot_unpack_bit_exact(rlx, scheme, path):
    M, N, K = PATHS[path]
    W = Weights(scheme, N, K, seed=9000 + 10 * SCHEMES.index(scheme) + sorted(PATHS).index(path))
    # every weight column is selected at least once: the few-row path needs K / M calls
    offsets = range(0, K, M) if M < K else [0]
    ulp_ok = path == "gemv" and scheme == "int4m"  # two fp32 roundings there (module docstring)
    for off in offsets:
        x, k = _one_hot_rows(M, K, off)
        got = W.run(rlx, x).view(torch.int16).cpu().numpy().view(np.uint16)
        # + 0.0: the dot product's accumulator starts at +0, so a -0 weight (q = 0 under a
        # negative scale) gives +0 (IEEE: +0 + -0 = +0)
        want = _rne_bf16_bits((W.w[:, k].T + 0.0).astype(np.float32))
        if ulp_ok:
            diff = np.abs(got.astype(np.int32) - want.astype(np.int32))
            assert diff.max() <= 1, f"{scheme} {path}: {np.count_nonzero(diff > 1)} outputs off by more than 1 ulp"
            continue
        bad = np.nonzero(got != want)
        assert bad[0].size == 0, (
            f"{scheme} {path} offset {off}: {bad[0].size} of {got.size} outputs differ; first at (m={bad[0][0]}, "
            f"n={bad[1][0]}, k={k[bad[0][0]]}): got {int(got[bad[0][0], bad[1][0]]):#06x} want "
            f"{int(want[bad[0][0], bad[1][0]]):#06x}")


@pytest.mark.parametrize("scheme", ["int8", "int4"])
@pytest.mark.parametrize("path", ["reg128x128", "dma64x64", "gemv"])
def test_one_hot_f32_output(rlx, scheme, path):
    """f32 output: the exact dequantised weight, except that the tiled int4
    path rounds each weight to bf16 before the product."""
    M, N, K = PATHS[path]
    W = Weights(scheme, N, K, seed=7 + len(path))
    x, k = _one_hot_rows(M, K, 3)
    got = W.run(rlx, x, out_dtype=torch.float32).cpu().numpy()
    assert got.dtype == np.float32
    want = W.w[:, k].T.astype(np.float32)
    if scheme == "int4" and path != "gemv":
        want = to_bf16_exact(want)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("scheme", ["int8", "int4"])
@pytest.mark.parametrize("epi", EPIS)
@pytest.mark.parametrize("N", [1152, 1536])
def test_quant_full_size_tile(rlx, scheme, epi, N):
    """M = 4096 selects the register-staged 128 x 128 tile for K = 384."""
    M, K = 4096, 384
    rng = np.random.default_rng(4000 + N + len(epi))
    W = Weights(scheme, N, K, seed=5000 + N)
    x = to_bf16_exact(rng.normal(0, 1, (M, K)))
    b = rng.normal(0, 0.5, N).astype(np.float32)
    r = to_bf16_exact(rng.normal(0, 1, (M, N)))
    got = W.run(rlx, x, bias=b, residual=r, epi=epi).float().cpu().numpy()
    ref = oracle.linear(x, W.w, None if epi == "none" else b)
    pre = None
    if epi == "gelu":
        pre, ref = ref, oracle.gelu(ref)
    if epi == "residual":
        ref = ref + r
    wrel = 0.0 if scheme == "int8" else 2.0 ** -9
    tol = gemm_tolerance(x, W.w, ref, out_bf16=True, weight_rel=wrel, pre=pre)
    if scheme == "int8":
        tol = tol + 2.0 ** -24 * np.abs(ref) * 4
    assert_within(got, ref, tol, f"{scheme} {epi} {M}x{N}x{K}")


@pytest.mark.parametrize("epi", EPIS)
def test_dense_bf16_full_size_tile(rlx, epi):
    """M = 16384 selects the dense bf16 128 x 128 tile."""
    M, N, K = 16384, 1152, 384
    rng = np.random.default_rng(6000 + len(epi))
    x = to_bf16_exact(rng.normal(0, 1, (M, K)))
    w = to_bf16_exact(rng.normal(0, 0.05, (N, K)))
    b = rng.normal(0, 0.5, N).astype(np.float32)
    r = to_bf16_exact(rng.normal(0, 1, (M, N)))
    y = rlx.dequant_matmul(_dev(x, torch.bfloat16), _dev(w, torch.bfloat16), bias=_dev(b, torch.float32),
                           residual=_dev(r, torch.bfloat16), epi=_epi_code(rlx, epi))
    got = y.float().cpu().numpy()
    ref = oracle.linear(x, w, None if epi == "none" else b)
    pre = None
    if epi == "gelu":
        pre, ref = ref, oracle.gelu(ref)
    if epi == "residual":
        ref = ref + r
    assert_within(got, ref, gemm_tolerance(x, w, ref, out_bf16=True, pre=pre), f"dense bf16 {epi} {M}x{N}x{K}")


@pytest.mark.parametrize("epi", EPIS)
@pytest.mark.parametrize("case", ["dense_dma", "int8_reg", "int4_dma", "int4_gemv"])
def test_f32_output_elementwise(rlx, case, epi):
    """bf16 activations, f32 output and f32 residual, against the oracle."""
    shapes = {"dense_dma": (300, 1152, 384), "int8_reg": (300, 384, 384), "int4_dma": (200, 384, 1536),
              "int4_gemv": (9, 384, 1024)}
    M, N, K = shapes[case]
    rng = np.random.default_rng(7000 + M + N + len(epi))
    x = to_bf16_exact(rng.normal(0, 1, (M, K)))
    b = rng.normal(0, 0.5, N).astype(np.float32)
    r = rng.normal(0, 1, (M, N)).astype(np.float32)
    if case == "dense_dma":
        w = to_bf16_exact(rng.normal(0, 0.05, (N, K)))
        y = rlx.dequant_matmul(_dev(x, torch.bfloat16), _dev(w, torch.bfloat16), bias=_dev(b, torch.float32),
                               residual=_dev(r, torch.float32), epi=_epi_code(rlx, epi), out_dtype=torch.float32)
        wrel = 0.0
    else:
        W = Weights(case.split("_")[0], N, K, seed=8000 + M)
        w = W.w
        y = W.run(rlx, x, bias=b, residual=r, epi=epi, out_dtype=torch.float32)
        wrel = 2.0 ** -9 if case == "int4_dma" else 0.0
    assert y.dtype == torch.float32
    got = y.cpu().numpy()
    ref = oracle.linear(x, w, None if epi == "none" else b)
    pre = None
    if epi == "gelu":
        pre, ref = ref, oracle.gelu(ref)
    if epi == "residual":
        ref = ref + r
    tol = gemm_tolerance(x, w, ref, out_bf16=False, weight_rel=wrel, pre=pre) + 2.0 ** -24 * np.abs(ref) * 4
    if case == "int4_gemv":
        # the few-row int4 bound of tests/test_gpu_gemv.py: 2^-9 sum_k |x_k| s_group(k)
        s_k = np.repeat(W.scales.astype(np.float64), 32, axis=1)
        tol = tol + 2.0 ** -9 * (np.abs(x.astype(np.float64)) @ s_k.T)
    assert_within(got, ref, tol, f"f32 output {case} {epi} {M}x{N}x{K}")
