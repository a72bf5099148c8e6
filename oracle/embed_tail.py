"""Op_embed's tail, fused with Op_upsert.  Test infrastructure only.

Section 4.3 turns each chunk into a vector as tokenize -> hidden states -> mean pool -> L2
normalise, and the vectors then go into the index (Op_upsert, Section 3.2).  The reading
used here:

* hidden states [m x T x h] with the chunk's first len tokens valid (right padding, len
  clamped to [0, T]); the mean is over those tokens;
* the embedding is mean / ||mean||_2, and the zero vector when len = 0 or the mean is 0;
* the vector is then stored like any upserted fp32 row (round to nearest even to the index
  dtype).

In exact arithmetic mean / ||mean|| = sum / ||sum||; the oracle forms the mean first, in fp64.
"""
from __future__ import annotations

import numpy as np


def pool(hidden64: np.ndarray, lengths) -> np.ndarray:
    """fp64 embeddings [m x h] of hidden states [m x T x h]."""
    H = np.asarray(hidden64, dtype=np.float64)
    m, T, h = H.shape
    out = np.zeros((m, h), dtype=np.float64)
    for i in range(m):
        n = int(min(max(int(lengths[i]), 0), T))
        if n == 0:
            continue
        mean = H[i, :n].mean(axis=0)
        nrm = float(np.sqrt((mean * mean).sum()))
        if nrm > 0:
            out[i] = mean / nrm
    return out
