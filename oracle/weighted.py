"""Weighted score fusion over the whole corpus.  Test infrastructure only.

Section 4.4 fuses dense and lexical evidence as score(d, q) = w_d s^_dense(d, q) +
w_l s^_lexical(d, q) over every chunk and takes the top k.  It names neither the
normalisation s^ nor the weights; the reading used here:

* s^ = per-query min-max normalisation over all N chunks, (s - min) / (max - min), and 0 for
  every chunk when max == min (a query with no lexical match, or a constant dense row);
* s_dense = the inner product (as the dense oracle), s_lexical = full-corpus BM25 (as the
  BM25 oracle; chunks without a matching term score 0 and take part in min and max);
* default weights w_d = w_l = 0.5; top k by (score desc, id asc).
"""
from __future__ import annotations

import numpy as np

from oracle import dense as od


def normalise(S: np.ndarray) -> np.ndarray:
    """Row-wise min-max normalisation in fp64; rows with max == min become 0."""
    S = np.asarray(S, dtype=np.float64)
    lo = S.min(axis=1, keepdims=True)
    hi = S.max(axis=1, keepdims=True)
    span = hi - lo
    out = np.zeros_like(S)
    ok = span[:, 0] > 0
    out[ok] = (S[ok] - lo[ok]) / span[ok]
    return out


def fused(S_dense: np.ndarray, S_lex: np.ndarray, w_d: float = 0.5, w_l: float = 0.5) -> np.ndarray:
    return w_d * normalise(S_dense) + w_l * normalise(S_lex)


def topk(S_dense, S_lex, k: int, w_d: float = 0.5, w_l: float = 0.5):
    """(ids [nq x k], fused scores [nq x k]) by (score desc, id asc)."""
    return od.topk_from_scores(fused(S_dense, S_lex, w_d, w_l), k)
