"""Reciprocal rank fusion in exact rational arithmetic.  Test infrastructure only.

The hybrid workload fuses a dense and a sparse ranked list with reciprocal rank fusion
(Cormack, Clarke and Buettcher, SIGIR 2009): fused(d) = sum over the lists L containing d of
1 / (k_rrf + rank_L(d)), ranks 1-based; a list that does not contain d adds nothing.  The
fused list is sorted by (fused desc, id asc) and cut at k.  Fractions keep exact ties exact
(1/63 = 2/126: rank 3 in one list ties rank 66 in both).
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np


def fuse_one(lists, rrf_k: int, k: int):
    """lists: iterable of id sequences (id -1 = empty slot, skipped without consuming a rank).

    Returns (ids [k] with -1 padding, fused Fractions [k] with None padding).
    """
    fused: dict[int, Fraction] = {}
    for lst in lists:
        rank = 0
        for d in lst:
            d = int(d)
            if d < 0:
                continue
            rank += 1
            fused[d] = fused.get(d, Fraction(0)) + Fraction(1, rrf_k + rank)
    order = sorted(fused.items(), key=lambda kv: (-kv[1], kv[0]))[:k]
    ids = [d for d, _ in order] + [-1] * (k - len(order))
    vals = [v for _, v in order] + [None] * (k - len(order))
    return ids, vals


def to_f32(v) -> np.float32:
    """fp32 of an exact fraction: nearest double (Fraction -> float), then nearest fp32."""
    return np.float32(-np.inf) if v is None else np.float32(float(v))


def fuse(dense_ids: np.ndarray, sparse_ids: np.ndarray, rrf_k: int, k: int):
    """Batch RRF: returns (ids int64 [B x k], fused fp32 [B x k], fused Fractions)."""
    dense_ids = np.atleast_2d(dense_ids)
    sparse_ids = np.atleast_2d(sparse_ids)
    B = dense_ids.shape[0]
    ids = np.full((B, k), -1, dtype=np.int64)
    f32 = np.full((B, k), -np.inf, dtype=np.float32)
    fr = []
    for q in range(B):
        i, v = fuse_one((dense_ids[q], sparse_ids[q]), rrf_k, k)
        ids[q] = i
        f32[q] = [to_f32(x) for x in v]
        fr.append(v)
    return ids, f32, fr
