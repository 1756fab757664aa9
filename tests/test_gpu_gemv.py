"""GPU parity of the few-row dequantising matmul (the GEMV regime of
rlx_dequant_matmul: int8 / int4 weights, 1 <= M <= 16 bf16 rows, K a multiple
of 128, M * K * 2 <= 64 KB), through the C ABI, against the CPU oracle on the
same dequantised weights.

Tolerances, from the arithmetic of the kernel:
* int8: the codes enter the matrix cores exactly and the scale multiplies the
  fp32 sum, as in the tiled path: fp32 accumulation, a few roundings of the
  scaled sum, bf16 output rounding.
* int4: no weight is rounded.  A group's instruction sums x_k (128 + q_k) in
  fp32 and the kernel subtracts s (128 + z) X with X the fp32 group sum of x:
  each of the two terms is off by at most 31 * 2^-24 * 143 * s sum_g |x_k|
  (< 2^-11.9 s sum_g |x_k|), and the accumulator, which holds up to four
  groups' 143 s X terms before they cancel, adds a few 2^-24 of that per
  group.  The bound used is 2^-9 sum_k |x_k| s_{group(k)}, over twice the sum
  of those terms, on top of the fp32 accumulation and bf16 output bounds.
"""
import numpy as np
import pytest

import oracle
import workloads
from gpu_helpers import assert_within, gemm_tolerance, to_bf16_exact

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

EPIS = ["none", "bias", "gelu", "residual"]


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


def _oracle(x, w, b, res, epi):
    y = oracle.linear(x, w, None if epi == "none" else b)
    if epi == "gelu":
        y = oracle.gelu(y)
    if epi == "residual":
        y = y + res
    return y


class Case:
    """Seeded inputs of one product: bf16 x [M, K], N(0, 0.02) weights quantised
    with the scheme, f32 bias N(0, 0.5), bf16 residual N(0, 1)."""

    def __init__(self, scheme, M, N, K, seed, zero_shift=0.0):
        rng = np.random.default_rng(seed)
        self.scheme, self.M, self.N, self.K = scheme, M, N, K
        self.x = to_bf16_exact(rng.normal(0, 1, (M, K)))
        wf = rng.normal(0, 0.02, (N, K)).astype(np.float32)
        self.b = rng.normal(0, 0.5, N).astype(np.float32)
        self.r = to_bf16_exact(rng.normal(0, 1, (M, N)))
        if scheme == "int8":
            self.q, self.s = workloads.quantize_int8_per_channel(wf)
            self.z = None
            self.wdeq = oracle.dequant_int8(self.q, self.s)
        else:
            self.q, self.s, self.z = workloads.quantize_int4_grouped(wf, 32)
            if zero_shift:  # zero-points off the integers (the layout allows any f16)
                self.z = (self.z.astype(np.float32) + np.float32(zero_shift)).astype(np.float16)
            self.wdeq = oracle.dequant_int4(self.q, self.s, self.z, 32)

    def run(self, rlx, epi, x=None):
        x = self.x if x is None else x
        kw = dict(N=self.N, bias=_dev(self.b, torch.float32), residual=_dev(self.r[:x.shape[0]], torch.bfloat16),
                  epi=_epi_code(rlx, epi))
        if self.scheme == "int8":
            y = rlx.dequant_matmul(_dev(x, torch.bfloat16), _dev(self.q, torch.int8), scheme=rlx.Q_INT8_PER_CHANNEL,
                                   scales=_dev(self.s, torch.float16), **kw)
        else:
            y = rlx.dequant_matmul(_dev(x, torch.bfloat16), _dev(self.q, torch.uint8), scheme=rlx.Q_INT4_GROUP_ZP,
                                   scales=_dev(self.s, torch.float16), zeros=_dev(self.z, torch.float16),
                                   group_size=32, **kw)
        torch.cuda.synchronize()
        return y

    def tolerance(self, ref, epi, cols=slice(None)):
        w = self.wdeq[cols]
        pre = oracle.linear(self.x, w, self.b[cols]) if epi == "gelu" else None
        tol = gemm_tolerance(self.x, w, ref, out_bf16=True, pre=pre)
        if self.scheme == "int8":
            return tol + 2.0 ** -24 * np.abs(ref) * 4  # scale applied to the fp32 sum
        s_k = np.repeat(self.s[cols].astype(np.float64), 32, axis=1)  # s of each weight's group
        return tol + 2.0 ** -9 * (np.abs(self.x.astype(np.float64)) @ s_k.T)


# (M, N, K): one row, ragged row counts, every N / K of the MiniLM encoder,
# K spanning 1 .. 32 units, and the 64 KB activation limit (M K = 32768)
SHAPES = [(1, 64, 128), (3, 1152, 384), (16, 1536, 384), (5, 384, 1536), (16, 256, 2048), (8, 512, 4096),
          (1, 4096, 4096)]


@pytest.mark.parametrize("scheme", ["int8", "int4"])
@pytest.mark.parametrize("epi", EPIS)
@pytest.mark.parametrize("M,N,K", SHAPES)
def test_gemv_parity(rlx, scheme, epi, M, N, K):
    c = Case(scheme, M, N, K, 4000 + 3 * M + N + K + (1 if scheme == "int4" else 0))
    got = c.run(rlx, epi).float().cpu().numpy()
    ref = _oracle(c.x, c.wdeq, c.b, c.r, epi)
    assert_within(got, ref, c.tolerance(ref, epi), f"gemv {scheme} {epi} {M}x{N}x{K}")


@pytest.mark.parametrize("shift", [0.375, -0.71875])
def test_int4_zero_points_off_the_integers(rlx, shift):
    c = Case("int4", 4, 512, 1024, 77, zero_shift=shift)
    got = c.run(rlx, "bias").float().cpu().numpy()
    ref = _oracle(c.x, c.wdeq, c.b, c.r, "bias")
    assert_within(got, ref, c.tolerance(ref, "bias"), f"int4 zero shift {shift}")


@pytest.mark.parametrize("scheme", ["int8", "int4"])
def test_rows_are_independent_and_results_repeat(rlx, scheme):
    """A row's result does not depend on the other rows in the call, and two
    calls give the same bits (the wave partials are added in a fixed order)."""
    c = Case(scheme, 11, 768, 1536, 91)
    full = c.run(rlx, "gelu").view(torch.int16).cpu().numpy()
    again = c.run(rlx, "gelu").view(torch.int16).cpu().numpy()
    assert np.array_equal(full, again)
    for m in (0, 5, 10):
        one = c.run(rlx, "gelu", x=c.x[m:m + 1]).view(torch.int16).cpu().numpy()
        assert np.array_equal(one[0], full[m]), m


@pytest.mark.parametrize("scheme", ["int8", "int4"])
@pytest.mark.parametrize("M", [1, 16])
def test_decode_shape_sampled_columns(rlx, scheme, M):
    """The benchmark's decode-sized product (N 14336, K 4096) on 96 sampled
    output columns (the oracle dequantises only those weight rows)."""
    N, K = 14336, 4096
    if M * K * 2 > 64 * 1024:
        M = 8  # the largest row count this K keeps in the few-row path
    rng = np.random.default_rng(5150 + M)
    x = to_bf16_exact(rng.normal(0, 1, (M, K)))
    wf = rng.normal(0, 0.02, (N, K)).astype(np.float32)
    b = rng.normal(0, 0.5, N).astype(np.float32)
    cols = np.sort(np.concatenate([rng.choice(N, 94, replace=False), [0, N - 1]]))
    if scheme == "int8":
        q, s = workloads.quantize_int8_per_channel(wf)
        y = rlx.dequant_matmul(_dev(x, torch.bfloat16), _dev(q, torch.int8), scheme=rlx.Q_INT8_PER_CHANNEL,
                               scales=_dev(s, torch.float16), N=N, bias=_dev(b, torch.float32), epi=rlx.EPI_BIAS)
        wdeq = oracle.dequant_int8(q[cols], s[cols])
        extra = None
    else:
        q, s, z = workloads.quantize_int4_grouped(wf, 32)
        y = rlx.dequant_matmul(_dev(x, torch.bfloat16), _dev(q, torch.uint8), scheme=rlx.Q_INT4_GROUP_ZP,
                               scales=_dev(s, torch.float16), zeros=_dev(z, torch.float16), group_size=32, N=N,
                               bias=_dev(b, torch.float32), epi=rlx.EPI_BIAS)
        wdeq = oracle.dequant_int4(q[cols], s[cols], z[cols], 32)
        extra = 2.0 ** -9 * (np.abs(x.astype(np.float64)) @ np.repeat(s[cols].astype(np.float64), 32, axis=1).T)
    torch.cuda.synchronize()
    got = y.float().cpu().numpy()[:, cols]
    ref = oracle.linear(x, wdeq, b[cols])
    tol = gemm_tolerance(x, wdeq, ref, out_bf16=True) + (2.0 ** -24 * 4 * np.abs(ref) if extra is None else extra)
    assert_within(got, ref, tol, f"decode shape {scheme} M={M}")


def test_rows_past_the_few_row_limit_take_the_tiled_path(rlx):
    """M = 16 with K = 4096 (128 KB of activations) and M = 17: the tiled path
    (each int4 weight rounded to bf16 before the product) gives the result."""
    for M, K in ((16, 4096), (17, 384)):
        c = Case("int4", M, 256, K, 600 + M)
        got = c.run(rlx, "residual").float().cpu().numpy()
        ref = _oracle(c.x, c.wdeq, c.b, c.r, "residual")
        tol = gemm_tolerance(c.x, c.wdeq, ref, out_bf16=True, weight_rel=2.0 ** -9)
        assert_within(got, ref, tol, f"tiled int4 {M}x{K}")
