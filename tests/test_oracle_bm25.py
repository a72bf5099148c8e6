"""Pins for the BM25 oracle: hand values, closed forms, a per-document pure-Python formulation
and the invariants of the BM25 formula (no GPU)."""
import math
from collections import Counter

import numpy as np
import pytest

import synth
from oracle import bm25


def _corpus(docs):
    indptr = np.zeros(len(docs) + 1, dtype=np.int64)
    indptr[1:] = np.cumsum([len(d) for d in docs])
    toks = np.array([t for d in docs for t in d], dtype=np.int32)
    return indptr, toks


def _queries(qs):
    ind = np.zeros(len(qs) + 1, dtype=np.int32)
    ind[1:] = np.cumsum([len(q) for q in qs])
    return ind, np.array([t for q in qs for t in q], dtype=np.int32)


def test_hand_example(load_golden):
    g = load_golden("bm25_hand.yaml")
    ind, toks = _corpus(g["docs"])
    qi, qt = _queries([q["terms"] for q in g["queries"]])
    S = bm25.scores_batch(ind, toks, qi, qt, g["k1"], g["b"])
    for r, q in enumerate(g["queries"]):
        np.testing.assert_allclose(S[r], q["scores"], rtol=0, atol=0.6 * 10 ** -g["digits"])
    idf = bm25.idf(3, np.array([2, 2, 1]))
    np.testing.assert_allclose(idf, [g["idf"][0], g["idf"][1], g["idf"][2]], rtol=1e-14)


def _py_bm25(docs, q, k1, b):
    """Independent per-document formulation with Counter and math.log."""
    n = len(docs)
    avgdl = math.fsum(len(d) for d in docs) / n
    cnt = [Counter(d) for d in docs]
    out = []
    for d, c in zip(docs, cnt):
        s = 0.0
        for t in q:
            df = sum(1 for cc in cnt if cc[t] > 0)
            w = math.log(1 + (n - df + 0.5) / (df + 0.5))
            tf = c[t]
            s += w * tf * (k1 + 1) / (tf + k1 * (1 - b + b * len(d) / avgdl))
        out.append(s)
    return out


def test_matches_per_document_formulation():
    rnd = np.random.default_rng(7)
    docs = [rnd.integers(0, 12, size=rnd.integers(1, 15)).tolist() for _ in range(40)]
    qs = [rnd.integers(0, 14, size=rnd.integers(1, 6)).tolist() for _ in range(25)]
    ind, toks = _corpus(docs)
    qi, qt = _queries(qs)
    S = bm25.scores_batch(ind, toks, qi, qt, 1.2, 0.75)
    for r, q in enumerate(qs):
        np.testing.assert_allclose(S[r], _py_bm25(docs, q, 1.2, 0.75), rtol=1e-13, atol=1e-15)


def test_closed_form_single_term_single_doc():
    # one chunk of length L with tf occurrences of term 0: df = 1, N = 1, dl = avgdl
    for L, tf in [(5, 2), (1, 1), (9, 9)]:
        docs = [[0] * tf + [1] * (L - tf)]
        ind, toks = _corpus(docs)
        qi, qt = _queries([[0]])
        s = bm25.scores_batch(ind, toks, qi, qt, 1.2, 0.75)[0, 0]
        # N - df + 0.5 = 0.5, df + 0.5 = 1.5 -> idf = ln(4/3); length norm = k1
        assert s == pytest.approx(math.log(4 / 3) * tf * 2.2 / (tf + 1.2), rel=1e-15)


def test_invariants():
    rnd = np.random.default_rng(8)
    docs = [rnd.integers(0, 20, size=rnd.integers(3, 30)).tolist() for _ in range(50)]
    ind, toks = _corpus(docs)
    qi, qt = _queries([[3, 5], [3], [3, 3]])
    S = bm25.scores_batch(ind, toks, qi, qt, 1.2, 0.75)
    has = np.array([(3 in d) or (5 in d) for d in docs])
    assert ((S[0] > 0) == has).all()                  # zero iff no query term
    np.testing.assert_allclose(S[2], 2 * S[1], rtol=1e-15)  # repeated term counts twice
    # b = 0 removes the length dependence; k1 = 0 gives sum of idf over present terms
    docs2 = [[0, 1, 2], [0, 1, 2, 3, 3, 3, 3], [0]]
    ind2, toks2 = _corpus(docs2)
    qi2, qt2 = _queries([[0]])
    s_b0 = bm25.scores_batch(ind2, toks2, qi2, qt2, 1.2, 0.0)[0]
    assert s_b0[0] == s_b0[1] == s_b0[2]
    s_k0 = bm25.scores_batch(ind2, toks2, qi2, qt2, 0.0, 0.75)[0]
    np.testing.assert_allclose(s_k0, bm25.idf(3, np.array([3]))[0], rtol=1e-15)
    # monotone: more occurrences at equal length scores higher; longer chunk at equal tf lower
    docs3 = [[0, 1, 1, 1], [0, 0, 1, 1], [0, 1, 1, 1, 1, 1, 1, 1], [2]]
    ind3, toks3 = _corpus(docs3)
    qi3, qt3 = _queries([[0]])
    s3 = bm25.scores_batch(ind3, toks3, qi3, qt3, 1.2, 0.75)[0]
    assert s3[1] > s3[0] > s3[2] > 0 and s3[3] == 0
    assert (bm25.idf(100, np.arange(1, 101)) > 0).all()


def test_k1_zero_absent_term_adds_nothing():
    # k1 = 0 makes the length norm 0; a chunk without the term must score 0, not 0/0
    ind, toks = _corpus([[0, 1], [1, 1], [2]])
    qi, qt = _queries([[0], [0, 1]])
    S = bm25.scores_batch(ind, toks, qi, qt, 0.0, 0.75)
    assert np.isfinite(S).all()
    idf0 = bm25.idf(3, np.array([1]))[0]
    idf1 = bm25.idf(3, np.array([2]))[0]
    np.testing.assert_allclose(S[0], [idf0, 0.0, 0.0], rtol=1e-15)
    np.testing.assert_allclose(S[1], [idf0 + idf1, idf1, 0.0], rtol=1e-15)


def test_sparse_topk_excludes_zero_and_orders_ties_by_id():
    S = np.array([[0.0, 2.0, 1.0, 2.0, 0.0, 0.5]])
    ids, sc = bm25.sparse_topk_from_scores(S, 6)
    assert ids[0].tolist() == [1, 3, 2, 5, -1, -1]
    assert np.isneginf(sc[0, 4:]).all()


def test_csr_layout_agrees_with_token_counts():
    """The generator's CSR (the library's input) carries the same tf / dl / df the oracle counts."""
    g = synth.rng(77, 3)
    ind, toks = synth.sparse_corpus(g, 300, 50, 1.1, 20.0)
    csr = synth.csr_from_tokens(ind, toks, 50)
    terms = np.arange(50)
    tf = bm25.term_frequencies(ind, toks, terms)
    for t in range(50):
        lo, hi = csr.term_indptr[t], csr.term_indptr[t + 1]
        docs = csr.post_chunk[lo:hi]
        assert (np.diff(docs) > 0).all()
        assert (tf[t, docs] == csr.post_tf[lo:hi]).all()
        assert np.count_nonzero(tf[t]) == hi - lo
    assert (csr.doc_len == np.diff(ind)).all()
