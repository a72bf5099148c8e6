"""BM25 by a document-wise scan of the raw token sequences.  Test infrastructure only.

Section 4.4 scores lexical relevance with BM25 and requires exact full-corpus semantics
(an inverted-postings implementation must give the same scores as scanning every
document).  The paper leaves the BM25 variant open; the reading used here:

* tf(t, d)  = occurrences of term t in chunk d;  dl(d) = token count of d;
* N = number of chunks;  avgdl = sum(dl) / N;  df(t) = #{d : tf(t, d) > 0};
* idf(t)    = ln(1 + (N - df + 0.5) / (df + 0.5))          (always positive);
* score(q, d) = sum over the term OCCURRENCES t of q that occur in d, in query order, of
      idf(t) * tf * (k1 + 1) / (tf + k1 * (1 - b + b * dl / avgdl));
  a term absent from d adds exactly 0 (this matters when k1 = 0, where the formula would
  read 0 / 0 for tf = 0).

Nothing here reads a postings list: term frequencies are counted from the token sequences.
"""
from __future__ import annotations

import numpy as np


def corpus_stats(doc_indptr: np.ndarray):
    """(N, dl fp64 [N], avgdl) of a corpus given by its token-sequence offsets."""
    dl = np.diff(np.asarray(doc_indptr, dtype=np.int64)).astype(np.float64)
    n = dl.shape[0]
    return n, dl, float(dl.sum()) / n


def term_frequencies(doc_indptr: np.ndarray, tokens: np.ndarray, terms: np.ndarray) -> np.ndarray:
    """tf[j, d] = number of occurrences of terms[j] in chunk d, counted over every token of every chunk."""
    terms = np.asarray(terms, dtype=np.int64)
    n = np.asarray(doc_indptr).shape[0] - 1
    doc_of_tok = np.repeat(np.arange(n, dtype=np.int64), np.diff(np.asarray(doc_indptr, dtype=np.int64)))
    tf = np.zeros((terms.shape[0], n), dtype=np.int64)
    if terms.shape[0] == 0:
        return tf
    slot = {int(t): j for j, t in enumerate(terms)}
    lut = np.full(int(max(terms.max(), np.max(tokens, initial=0))) + 1, -1, dtype=np.int64)
    for t, j in slot.items():
        lut[t] = j
    tok = np.asarray(tokens, dtype=np.int64)
    j_of_tok = lut[tok]
    hit = j_of_tok >= 0
    np.add.at(tf, (j_of_tok[hit], doc_of_tok[hit]), 1)
    return tf


def idf(n_docs: int, df: np.ndarray) -> np.ndarray:
    df = np.asarray(df, dtype=np.float64)
    return np.log(1.0 + (n_docs - df + 0.5) / (df + 0.5))


def scores_batch(doc_indptr, tokens, qterm_indptr, qterms, k1: float, b: float) -> np.ndarray:
    """fp64 BM25 scores [nq x N] for every query of a batch against every chunk."""
    qterm_indptr = np.asarray(qterm_indptr, dtype=np.int64)
    qterms = np.asarray(qterms, dtype=np.int64)
    n, dl, avgdl = corpus_stats(doc_indptr)
    uniq = np.unique(qterms)
    tf = term_frequencies(doc_indptr, tokens, uniq).astype(np.float64)   # [n_uniq x N]
    df = np.count_nonzero(tf, axis=0 if tf.shape[0] == 0 else 1)
    w_idf = idf(n, df)
    norm = k1 * (1.0 - b + b * dl / avgdl)                                # [N]
    row = {int(t): j for j, t in enumerate(uniq)}
    nq = qterm_indptr.shape[0] - 1
    out = np.zeros((nq, n), dtype=np.float64)
    for q in range(nq):
        for t in qterms[qterm_indptr[q]:qterm_indptr[q + 1]]:
            j = row[int(t)]
            f = tf[j]
            has = f > 0                     # a term absent from a chunk adds nothing to its score
            out[q, has] += w_idf[j] * f[has] * (k1 + 1.0) / (f[has] + norm[has])
    return out


def sparse_topk_from_scores(S: np.ndarray, k: int):
    """Per query: chunks with score > 0, full stable sort on (score desc, id asc), first k.

    Chunks that contain no query term score 0 and are not ranked; short lists are padded
    with id -1 and score -inf.
    """
    S = np.atleast_2d(np.asarray(S, dtype=np.float64))
    B, n = S.shape
    ids = np.full((B, k), -1, dtype=np.int64)
    sc = np.full((B, k), -np.inf, dtype=np.float64)
    for q in range(B):
        pos = np.flatnonzero(S[q] > 0.0)
        order = pos[np.argsort(-S[q, pos], kind="stable")][:k]
        ids[q, :order.shape[0]] = order
        sc[q, :order.shape[0]] = S[q, order]
    return ids, sc


def topk(doc_indptr, tokens, qterm_indptr, qterms, k: int, k1: float = 1.2, b: float = 0.75):
    return sparse_topk_from_scores(scores_batch(doc_indptr, tokens, qterm_indptr, qterms, k1, b), k)
