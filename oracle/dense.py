"""Dense exact top-k, by definition.  Test infrastructure only (see the package docstring).

Retrieval R_k = Op_retrieve(q, I) (Section 3.2, "Retrieval") returns the k indexed vectors
with the largest inner product with the query; dense scores are plain matrix products over
the embedding matrix (Section 4.4), and the stored vectors are unit-norm (the embedding
path ends in an L2 normalisation, Section 4.3).  The paper fixes no tie order; the reading
used everywhere here is (score descending, row id ascending).
"""
from __future__ import annotations

import numpy as np

from .storage import decode


def scores(rows64: np.ndarray, queries64: np.ndarray) -> np.ndarray:
    """S[q, i] = sum_j Q[q, j] * X[i, j] in fp64 (one library matmul)."""
    return np.asarray(queries64, dtype=np.float64) @ np.asarray(rows64, dtype=np.float64).T


def topk_from_scores(S: np.ndarray, k: int):
    """First k of a full stable sort of each row of S on (score desc, id asc).

    Returns (ids int64 [B x k], scores fp64 [B x k]); when k exceeds the number of rows the
    tail is padded with id -1 and score -inf.
    """
    S = np.atleast_2d(np.asarray(S, dtype=np.float64))
    B, n = S.shape
    order = np.argsort(-S, axis=1, kind="stable")  # stable: equal scores keep ascending ids
    kk = min(k, n)
    ids = np.full((B, k), -1, dtype=np.int64)
    sc = np.full((B, k), -np.inf, dtype=np.float64)
    ids[:, :kk] = order[:, :kk]
    sc[:, :kk] = np.take_along_axis(S, order[:, :kk], axis=1)
    return ids, sc


def topk(rows_bits: np.ndarray, queries_bits: np.ndarray, dtype: str, k: int):
    """Exact top-k of stored queries against stored rows (both given as raw bits)."""
    X = decode(rows_bits, dtype)
    Q = decode(queries_bits, dtype)
    return topk_from_scores(scores(X, Q), k)


def abs_dot(rows64: np.ndarray, queries64: np.ndarray) -> np.ndarray:
    """sum_j |Q[q, j] * X[i, j]|, the magnitude that bounds the rounding error of an fp32 sum."""
    return np.abs(np.asarray(queries64, dtype=np.float64)) @ np.abs(np.asarray(rows64, dtype=np.float64)).T
