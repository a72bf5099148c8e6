"""Pins for the weighted-fusion oracle: hand cases (tests/golden/weighted_hand.yaml, from the
BM25 hand values) and properties fixed by the definition: min-max normalisation maps each
row onto [0, 1] with min -> 0 and max -> 1 and ignores positive affine changes of the scores;
one weight at zero reduces to the other ranking; a constant row contributes nothing."""
import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import bm25, weighted
from oracle import dense as od


def _bm25(docs, terms, k1, b):
    ind = np.zeros(len(docs) + 1, dtype=np.int64)
    ind[1:] = np.cumsum([len(d) for d in docs])
    toks = np.array([t for d in docs for t in d], dtype=np.int64)
    qi = np.array([0, len(terms)], dtype=np.int64)
    return bm25.scores_batch(ind, toks, qi, np.array(terms, dtype=np.int64), k1, b)


def test_hand_cases(load_golden):
    g = load_golden("weighted_hand.yaml")
    S = np.array([g["dense"]], dtype=np.float64)
    for c in g["cases"]:
        B = _bm25(g["docs"], c["terms"], g["k1"], g["b"])
        ids, sc = weighted.topk(S, B, 3, *c["w"])
        assert ids[0].tolist() == c["ids"], c
        np.testing.assert_allclose(sc[0], c["scores"], rtol=0, atol=1e-12)


@settings(max_examples=80, deadline=None)
@given(st.integers(0, 10**6), st.floats(0.1, 10.0), st.floats(-5.0, 5.0))
def test_normalisation_range_and_affine_invariance(seed, scale, shift):
    g = np.random.default_rng(seed)
    S = g.normal(size=(3, 40))
    N = weighted.normalise(S)
    assert np.allclose(N.min(axis=1), 0) and np.allclose(N.max(axis=1), 1)
    assert np.allclose(weighted.normalise(scale * S + shift), N, atol=1e-12)
    assert np.array_equal(weighted.normalise(np.ones((2, 5))), np.zeros((2, 5)))


@settings(max_examples=60, deadline=None)
@given(st.integers(0, 10**6))
def test_one_weight_zero_reduces_to_one_ranking(seed):
    g = np.random.default_rng(seed)
    Sd = g.integers(-9, 9, size=(2, 30)).astype(np.float64)
    Sl = np.maximum(0, g.integers(-4, 9, size=(2, 30))).astype(np.float64)
    ids_d, _ = weighted.topk(Sd, Sl, 10, 1.0, 0.0)
    ref_d, _ = od.topk_from_scores(Sd, 10)
    assert np.array_equal(ids_d, ref_d)
    ids_l, _ = weighted.topk(Sd, Sl, 10, 0.0, 1.0)
    ref_l, _ = od.topk_from_scores(Sl, 10)
    assert np.array_equal(ids_l, ref_l)


def test_planted_mistake_fails(load_golden):
    """Normalising by the maximum alone (no subtraction of the minimum) changes the first hand
    case, so the hand pins would catch it."""
    g = load_golden("weighted_hand.yaml")
    S = np.array([g["dense"]], dtype=np.float64)
    c = g["cases"][0]
    B = _bm25(g["docs"], c["terms"], g["k1"], g["b"])
    wrong = 0.5 * S / S.max() + 0.5 * B / B.max()
    _, sc = od.topk_from_scores(wrong, 3)
    assert not np.allclose(sc[0], c["scores"], rtol=0, atol=1e-6)
