"""The attention benchmark's work accounting (CPU only): the visible (query,
key) pairs bench.py counts for its TFLOP/s figure equal the count of the
oracle's own visibility matrix, summed over the batch, for every mask kind."""
import numpy as np
import pytest

import bench
import oracle
from oracle.encoder import visible_keys

KINDS = {"none": oracle.MASK_NONE, "causal": oracle.MASK_CAUSAL, "sliding": oracle.MASK_SLIDING_WINDOW,
         "custom": oracle.MASK_CUSTOM}


@pytest.mark.parametrize("kind", sorted(KINDS))
@pytest.mark.parametrize("S,window", [(1, 1), (37, 5), (128, 128), (200, 300), (512, 128)])
def test_attention_pairs_match_the_oracle_visibility(kind, S, window):
    rng = np.random.default_rng(S + window)
    lens = np.concatenate([rng.integers(1, S + 1, 3), [S]])
    want = 0
    for L in lens:
        row = (np.arange(S) < L).astype(np.uint8) if kind == "custom" else None
        want += int(visible_keys(S, KINDS[kind], row, window).sum())
    assert bench.attention_pairs(kind, S, lens, window) == want


@pytest.mark.parametrize("scheme", ["int4", "int8", "q4_0", "q4_1", "q8_0"])
@pytest.mark.parametrize("M,N,K", [(1, 64, 128), (5, 192, 256)])
def test_gemv_bytes_match_the_buffers(scheme, M, N, K):
    """bench.py's algorithmic bytes of the few-row matmul equal the sizes of the
    buffers one call reads and writes: the weight codes and their per-channel
    or per-group metadata (GGUF schemes as their repacked layout: 4-bit codes
    two per byte or int8 codes, one f16 scale per 32-weight block, and one f16
    zero / min per block for the 4-bit ones), bf16 x and y, and the f32 bias."""
    import workloads
    from workloads import gguf as wg
    rng = np.random.default_rng(N + K)
    w = rng.normal(0, 0.02, (N, K)).astype(np.float32)
    if scheme == "int4":
        weight = sum(a.nbytes for a in workloads.quantize_int4_grouped(w, 32))
    elif scheme == "int8":
        weight = sum(a.nbytes for a in workloads.quantize_int8_per_channel(w))
    else:
        codes, d, m = oracle.gguf.parse(wg.quantize(w, scheme), scheme, K)
        per_code = 0.5 if scheme != "q8_0" else 1.0
        weight = int(codes.size * per_code) + 2 * d.size + (2 * d.size if scheme != "q8_0" else 0)
    io = 2 * M * K + 2 * M * N + 4 * N
    assert bench.gemv_bytes(scheme, M, N, K) == weight + io
