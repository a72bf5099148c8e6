"""Dense-first hybrid retrieval: lexical scoring of the dense candidates only.  Test
infrastructure only.

The paper's serving schedule (Section 4.1, "Retrieval", and the query-serving experiment of
Section 5.5) first takes a dense top-n candidate set and applies lexical reranking to those
candidates alone, then reports Recall@k and Jaccard overlap against full hybrid retrieval.
It names the schedule, not the formula; the reading used here:

* candidates = the exact dense top-n (ids, dense order = rank 1 .. n);
* a candidate's lexical score = its BM25 score over the whole corpus (idf, N and avgdl of
  every chunk, the definition in ``oracle.bm25``);
* the candidates with a positive lexical score are ranked by (score desc, id asc);
* reciprocal rank fusion (k_rrf) of the dense order of the candidates and that lexical
  order, cut at k by (fused desc, id asc) -- the fusion the full hybrid uses, so the two
  schedules differ only in which chunks compete.
"""
from __future__ import annotations

import numpy as np

from oracle import rrf


def lexical_order(cand_ids, lex_scores) -> list[int]:
    """Candidates with a positive lexical score, by (score desc, id asc)."""
    pairs = [(-float(s), int(i)) for i, s in zip(cand_ids, lex_scores) if int(i) >= 0 and s > 0]
    return [i for _, i in sorted(pairs)]


def rerank_one(cand_ids, lex_scores, rrf_k: int, k: int):
    """cand_ids in dense order (-1 = empty slot); lex_scores the candidates' BM25 scores.

    Returns (ids [k] with -1 padding, fused Fractions [k] with None padding)."""
    return rrf.fuse_one((list(cand_ids), lexical_order(cand_ids, lex_scores)), rrf_k, k)


def batch(cand_ids: np.ndarray, B: np.ndarray, rrf_k: int, k: int):
    """cand_ids [nq x n] dense candidates, B [nq x N] BM25 scores of every chunk.

    Returns (ids [nq x k] int64, fp32 fused [nq x k], exact Fractions)."""
    nq = cand_ids.shape[0]
    ids = np.full((nq, k), -1, dtype=np.int64)
    f32 = np.full((nq, k), -np.inf, dtype=np.float32)
    exact = []
    for q in range(nq):
        c = cand_ids[q]
        lex = [B[q, i] if i >= 0 else 0.0 for i in c]
        i_q, v_q = rerank_one(c, lex, rrf_k, k)
        ids[q] = i_q
        f32[q] = [rrf.to_f32(v) for v in v_q]
        exact.append(v_q)
    return ids, f32, exact
