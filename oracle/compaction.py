"""Token compaction maps (test infrastructure; see package docstring).

The paper's benchmark feeds padded batches to the encoder (Section VIII-B);
attention excludes masked keys, so no real token depends on a masked one, and
every row-local step can run on the real tokens alone.  The maps that list
them are index work with one correct answer, defined here plainly:

  L_b        = number of nonzero mask bytes of sequence b
  cu         = [0, L_0, L_0 + L_1, ...]                      (length B + 1)
  tok_src    = b*S + s of every real token (b, s), sequences in order,
               positions ascending                           (length cu[B])
  tok_dst    = for every (b, s) in row-major order, its index in tok_src,
               or -1 when masked                             (length B*S)
  order      = the sequence indices sorted by L_b, largest first, equal
               counts by index                                (length B)
"""
from __future__ import annotations

import numpy as np


def token_maps(mask):
    """mask [B, S] (nonzero = real token) -> (cu, tok_src, tok_dst, order), int64 arrays."""
    m = np.asarray(mask) != 0
    B, S = m.shape
    lengths = m.sum(axis=1)
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    tok_src = np.flatnonzero(m.reshape(-1)).astype(np.int64)  # row-major order = sequences, then positions
    tok_dst = np.full(B * S, -1, dtype=np.int64)
    tok_dst[tok_src] = np.arange(tok_src.size)
    order = np.lexsort((np.arange(B), -lengths)).astype(np.int64)  # primary key: -L; ties: index
    return cu, tok_src, tok_dst, order
