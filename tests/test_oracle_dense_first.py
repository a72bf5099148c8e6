"""Pins for the dense-first hybrid oracle: hand cases (tests/golden/dense_first_hand.yaml,
from the BM25 and RRF hand values), and properties that fix it independently of its code:
with every chunk a candidate it equals full hybrid retrieval over full-length lists; every
returned id is a dense candidate; a candidate with no lexical match keeps its dense-only
fused value; and pruning never adds a chunk the full schedule ranks lower."""
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import bm25, dense_first, rrf
from oracle import dense as od


def _bm25(docs, terms, k1, b):
    ind = np.zeros(len(docs) + 1, dtype=np.int64)
    ind[1:] = np.cumsum([len(d) for d in docs])
    toks = np.array([t for d in docs for t in d], dtype=np.int64)
    qi = np.array([0, len(terms)], dtype=np.int64)
    return bm25.scores_batch(ind, toks, qi, np.array(terms, dtype=np.int64), k1, b)[0]


def test_hand_cases(load_golden):
    g = load_golden("dense_first_hand.yaml")
    S = np.array([g["dense"]], dtype=np.float64)
    for c in g["cases"]:
        B = _bm25(g["docs"], c["terms"], g["k1"], g["b"])
        cand, _ = od.topk_from_scores(S, c["n_cand"])
        ids, vals = dense_first.rerank_one(cand[0], B[cand[0]], 60, c["k"])
        assert ids == c["ids"], c
        assert vals == [None if v is None else Fraction(v) for v in c["fused"]], c


def _random_case(seed, n_docs=30, vocab=12):
    g = np.random.default_rng(seed)
    docs = [list(g.integers(0, vocab, size=g.integers(0, 9))) for _ in range(n_docs)]
    terms = list(g.integers(0, vocab, size=g.integers(1, 5)))
    S = g.integers(-20, 20, size=(1, n_docs)).astype(np.float64)   # ties on purpose
    return docs, terms, S, _bm25(docs, terms, 1.2, 0.75)


@settings(max_examples=60, deadline=None)
@given(st.integers(0, 10**6))
def test_all_candidates_equal_full_hybrid(seed):
    docs, terms, S, B = _random_case(seed)
    n = len(docs)
    cand, _ = od.topk_from_scores(S, n)
    full_sparse = [i for i in bm25.sparse_topk_from_scores(B[None, :], n)[0][0] if i >= 0]
    ids_full, vals_full = rrf.fuse_one((list(cand[0]), full_sparse), 60, 10)
    ids, vals = dense_first.rerank_one(cand[0], B[cand[0]], 60, 10)
    assert ids == ids_full and vals == vals_full


@settings(max_examples=60, deadline=None)
@given(st.integers(0, 10**6), st.integers(1, 12))
def test_outputs_are_candidates_and_dense_only_values(seed, n_cand):
    docs, terms, S, B = _random_case(seed)
    cand, _ = od.topk_from_scores(S, n_cand)
    c = list(cand[0])
    ids, vals = dense_first.rerank_one(c, B[c], 60, 8)
    lex = dense_first.lexical_order(c, B[c])
    for i, v in zip(ids, vals):
        if i < 0:
            assert v is None
            continue
        assert i in c
        expect = Fraction(1, 60 + c.index(i) + 1)
        if B[i] > 0:
            expect += Fraction(1, 60 + lex.index(i) + 1)
        assert v == expect
    # sorted by (fused desc, id asc) and padded only past the candidates
    real = [(v, i) for i, v in zip(ids, vals) if i >= 0]
    assert real == sorted(real, key=lambda t: (-t[0], t[1]))
    assert len(real) == min(8, len(c))


def test_planted_mistake_fails(load_golden):
    """Dropping the lexical restriction to the candidates (ranking lexically over the whole
    corpus) changes the first hand case, so the hand pins would catch it."""
    g = load_golden("dense_first_hand.yaml")
    c = g["cases"][0]
    B = _bm25(g["docs"], c["terms"], g["k1"], g["b"])
    cand = [1, 2]
    wrong = rrf.fuse_one((cand, dense_first.lexical_order([0, 1, 2], B)), 60, c["k"])[0]
    assert wrong != c["ids"]
