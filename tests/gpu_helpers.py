"""Shared helpers of the GPU parity tests (tolerances derived from the arithmetic)."""
import numpy as np

BF16_REL = 2.0 ** -8   # RNE to bf16: relative error <= 2^-9 of the value; 2^-8 bounds it with slack
F32_EPS = 2.0 ** -24


def to_bf16_exact(a):
    """fp32 -> bf16-representable fp32 (inputs only)."""
    import workloads
    return workloads.round_to_bf16(np.asarray(a, np.float32))


# The GELU epilogue evaluates erf with Abramowitz & Stegun 7.1.28 (|error| <= 3e-7)
# in fp32: GELU(v) = v/2 (1 + erf(v / sqrt 2)) is then off by at most
# |v|/2 * (3e-7 + a few fp32 roundings) <= 5e-7 |v|.
GELU_REL = 5e-7


def gemm_tolerance(x, w, ref, *, out_bf16, weight_rel=0.0, pre=None):
    """Per-element bound for y = x W^T (+ epilogue) computed in fp32 from exact
    operands: fp32 accumulation (K * 2^-24 * sum|x||w|), optional relative
    weight rounding (weight_rel * sum|x||w|), bf16 output rounding
    (2^-8 * |ref|), the GELU approximation (GELU_REL * |pre-activation|) when
    `pre` is given, and a small floor."""
    ax = np.abs(np.asarray(x, np.float64))
    aw = np.abs(np.asarray(w, np.float64))
    s1 = ax @ aw.T
    K = ax.shape[1]
    tol = (K * F32_EPS + weight_rel) * s1 + 1e-6 * np.abs(ref) + 1e-6
    if pre is not None:
        tol = tol + GELU_REL * np.abs(pre)
    if out_bf16:
        tol = tol + BF16_REL * np.abs(ref)
    return tol


def assert_within(got, ref, tol, what=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    bad = err > tol
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    if bad.any():
        i = np.unravel_index(np.argmax(err - tol), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} elements out of tolerance; worst at {i}: "
                             f"got {got[i]!r} ref {ref[i]!r} err {err[i]:.3g} tol {np.broadcast_to(tol, err.shape)[i]:.3g}")
