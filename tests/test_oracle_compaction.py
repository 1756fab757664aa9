"""Pins of oracle.compaction: a hand-worked mask, and pure-Python loops over
positions on random small masks (an independent restatement: counters walked
token by token, the order by repeated selection of the longest remaining
sequence)."""
import numpy as np

import oracle


def _loops(mask):
    B, S = len(mask), len(mask[0])
    cu, src, dst = [0], [], []
    for b in range(B):
        for s in range(S):
            if mask[b][s]:
                dst.append(len(src))
                src.append(b * S + s)
            else:
                dst.append(-1)
        cu.append(len(src))
    counts = [cu[b + 1] - cu[b] for b in range(B)]
    left, order = list(range(B)), []
    while left:
        best = left[0]
        for b in left:
            if counts[b] > counts[best]:
                best = b
        order.append(best)
        left.remove(best)
    return cu, src, dst, order


def test_hand_worked_mask():
    mask = np.array([[1, 1, 0, 0], [0, 0, 0, 0], [1, 0, 1, 1], [1, 1, 0, 0]], np.uint8)
    cu, src, dst, order = oracle.compaction.token_maps(mask)
    assert cu.tolist() == [0, 2, 2, 5, 7]
    assert src.tolist() == [0, 1, 8, 10, 11, 12, 13]
    assert dst.tolist() == [0, 1, -1, -1, -1, -1, -1, -1, 2, -1, 3, 4, 5, 6, -1, -1]
    assert order.tolist() == [2, 0, 3, 1]  # 3 tokens, then the two of 2 by index, then the empty one


def test_against_position_loops():
    rng = np.random.default_rng(5)
    for _ in range(40):
        B, S = int(rng.integers(1, 9)), int(rng.integers(1, 12))
        mask = (rng.random((B, S)) < rng.random()).astype(np.uint8) * rng.integers(1, 256, (B, S)).astype(np.uint8)
        got = oracle.compaction.token_maps(mask)
        want = _loops(mask.tolist())
        for g, w in zip(got, want):
            assert g.tolist() == list(w)
