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
