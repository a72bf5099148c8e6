"""Pins for the RRF oracle (hand values, order consistency, symmetry) and for the acceptance
rules (they accept exact results and near-tie swaps, and reject planted mistakes)."""
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import accept, rrf


def test_hand_cases(load_golden):
    for c in load_golden("rrf_hand.yaml")["cases"]:
        ids, vals = rrf.fuse_one((c["dense"], c["sparse"]), 60, c["k"])
        assert ids == c["ids"]
        assert vals == [Fraction(v) for v in c["fused"]]


def test_tie_rank66_vs_rank3():
    # 2/126 == 1/63: id 9 at rank 3 of one list ties id 4 at rank 66 of both lists
    dense = list(range(100, 102)) + [9] + list(range(200, 262)) + [4]
    sparse = list(range(300, 365)) + [4]
    ids, vals = rrf.fuse_one((dense, sparse), 60, 200)
    assert vals[ids.index(4)] == vals[ids.index(9)] == Fraction(1, 63)
    assert ids.index(4) < ids.index(9)


def test_single_list_keeps_order_and_padding():
    ids, vals = rrf.fuse_one(([5, 2, 8, -1], [-1, -1]), 60, 5)
    assert ids == [5, 2, 8, -1, -1]
    assert vals[:3] == [Fraction(1, 61), Fraction(1, 62), Fraction(1, 63)] and vals[3] is None
    assert rrf.to_f32(vals[0]) == np.float32(1 / 61) and np.isneginf(rrf.to_f32(None))


lists = st.lists(st.integers(0, 40), min_size=0, max_size=25, unique=True)


@settings(max_examples=150, deadline=None)
@given(lists, lists)
def test_symmetry_and_order_consistency(a, b):
    i1, v1 = rrf.fuse_one((a, b), 60, 60)
    i2, v2 = rrf.fuse_one((b, a), 60, 60)
    assert i1 == i2 and v1 == v2
    inf = 10 ** 9
    rank = lambda lst, d: lst.index(d) if d in lst else inf
    pos = {d: r for r, d in enumerate(i1) if d >= 0}
    for x in pos:
        for y in pos:
            if rank(a, x) <= rank(a, y) and rank(b, x) <= rank(b, y) and x != y:
                assert v1[pos[x]] >= v1[pos[y]]


# ---------------------------------------------------------------- acceptance rules

def _s():
    # scores with a near-tie pair (ids 3, 4) and well separated others
    return np.array([0.10, 0.90, 0.50, 0.700000, 0.7000004, 0.20, 0.30])


def test_accepts_exact_and_near_tie_swap():
    s = _s()
    ids = np.array([1, 4, 3, 2])
    rep = accept.check_ranked(s, ids, s[ids].astype(np.float32), 4, rtol=2e-3)
    assert rep.ok, rep.problems
    swapped = np.array([1, 3, 4, 2])
    # GPU saw 3 and 4 equal in fp32 -> id order
    sc = np.array([0.9, 0.7, 0.7, 0.5], np.float32)
    rep = accept.check_ranked(s, swapped, sc, 4, rtol=2e-3)
    assert rep.ok and rep.n_subst == 2 and rep.recall == 1.0, rep.problems


@pytest.mark.parametrize("ids,scores,why", [
    ([1, 4, 2, 3], [0.9, 0.7000004, 0.5, 0.7], "isolated row out of place"),
    ([1, 4, 3, 6], [0.9, 0.7000004, 0.7, 0.3], "missed row"),
    ([1, 4, 3, 2], [0.9, 0.7000004, 0.7, 0.51], "score parity"),
    ([1, 4, 3, 3], [0.9, 0.7000004, 0.7, 0.7], "repeated id"),
    ([1, 4, 3, -1], [0.9, 0.7000004, 0.7, -np.inf], "short list"),
    ([4, 1, 3, 2], [0.7000004, 0.9, 0.7, 0.5], "unordered"),
])
def test_rejects_planted_mistakes(ids, scores, why):
    s = _s()
    rep = accept.check_ranked(s, np.array(ids), np.array(scores), 4, rtol=2e-3)
    assert not rep.ok, why


def test_strict_mode_uses_error_bounds():
    s = np.array([0.5, 0.5 + 1e-9, 0.2])
    err = np.array([1e-8, 1e-8, 1e-8])
    rep = accept.check_ranked(s, np.array([0, 1]), np.array([0.5, 0.5]), 2, mode="strict", err=err)
    assert rep.ok, rep.problems
    err = np.array([1e-12, 1e-12, 1e-12])
    rep = accept.check_ranked(s, np.array([0, 1]), np.array([0.5, 0.5]), 2, mode="strict", err=err)
    assert not rep.ok


def test_ranked_mask_and_padding():
    s = np.array([0.0, 2.0, 0.0, 1.0])
    ranked = s > 0
    rep = accept.check_ranked(s, np.array([1, 3, -1]), np.array([2.0, 1.0, -np.inf]), 3, rtol=1e-5, ranked=ranked)
    assert rep.ok, rep.problems
    rep = accept.check_ranked(s, np.array([1, 3, 0]), np.array([2.0, 1.0, 0.0]), 3, rtol=1e-5, ranked=ranked)
    assert not rep.ok


def _cert(ids, scores, k=3, n_rows=100, s_un=None):
    s_ret = np.array([0.9, 0.8, 0.7])
    return accept.certificate(s_ret, np.array(ids), np.array(scores, dtype=np.float64), np.full(3, 1e-6), k, n_rows,
                              s_unreturned=s_un, err_unreturned=None if s_un is None else np.full(len(s_un), 1e-6))


def test_certificate_accepts_complete_list():
    assert _cert([5, 2, 9], [0.9, 0.8, 0.7], s_un=[0.69, 0.5]).ok
    # fewer rows than k: the valid prefix is min(k, n_rows), then padding
    rep = accept.certificate(np.array([0.9, 0.8, 0.0]), np.array([1, 0, -1]), np.array([0.9, 0.8, -np.inf]),
                             np.full(3, 1e-6), 3, 2)
    assert rep.ok, rep.problems


@pytest.mark.parametrize("ids,scores,s_un,why", [
    ([5, 2, -1], [0.9, 0.8, -np.inf], None, "truncated list"),
    ([-1, -1, -1], [-np.inf] * 3, None, "empty list"),
    ([5, -1, 9], [0.9, -np.inf, 0.7], None, "hole in the prefix"),
    ([5, 2, 100], [0.9, 0.8, 0.7], None, "id past the rows"),
    ([5, 5, 9], [0.9, 0.8, 0.7], None, "repeated id"),
    ([5, 2, 9], [0.9, 0.8, 0.71], None, "score parity"),
    ([2, 5, 9], [0.8, 0.9, 0.7], None, "unordered"),
    ([5, 2, 9], [0.9, 0.8, 0.7], [0.3, 0.7001], "missed row"),
])
def test_certificate_rejects_planted_mistakes(ids, scores, s_un, why):
    assert not _cert(ids, scores, s_un=s_un).ok, why


def test_strict_bound_covers_fp32_sums():
    """The per-row bound 2 gamma_d sum|q x| holds for fp32 recursive sums of the exact products
    in forward, reverse and pairwise-blocked orders (rounded products included)."""
    g = np.random.default_rng(3)
    for d in (64, 384, 1024):
        X = g.standard_normal((40, d)).astype(np.float32)
        q = g.standard_normal(d).astype(np.float32)
        exact = X.astype(np.float64) @ q.astype(np.float64)
        bound = accept.strict_err(np.abs(X.astype(np.float64)) @ np.abs(q.astype(np.float64)), d)
        for order in (np.arange(d), np.arange(d)[::-1], g.permutation(d)):
            acc = np.zeros(40, np.float32)
            for j in order:
                acc = acc + X[:, j] * q[j]  # fp32 product, then fp32 add
            assert np.all(np.abs(acc.astype(np.float64) - exact) <= bound)
        blocked = (X.reshape(40, -1, 32) * q.reshape(-1, 32)).sum(axis=2, dtype=np.float32).sum(axis=1, dtype=np.float32)
        assert np.all(np.abs(blocked.astype(np.float64) - exact) <= bound)


# ---------------------------------------------------------------- dense-first acceptance

def _df_case():
    # dense order 10..14; lexical: 14 first, 11 second, 12 and 13 within the fp32 bound
    cand = [10, 11, 12, 13, 14, -1]
    lex = np.array([0.0, 5.0, 3.0, 3.0 + 1e-9, 7.0, 0.0])
    return cand, lex, accept.bm25_f32_err(lex, 8)


def _f(*vals):
    return np.array([np.float32(float(v)) for v in vals], dtype=np.float32)


def test_dense_first_accepts_both_readings_of_a_near_tie():
    cand, lex, err = _df_case()
    F = Fraction
    # 13 above 12 (the fp64 order): 12 = 1/63 + 1/64 ties 13 = 1/64 + 1/63, id order
    exact = accept.check_dense_first(cand, lex, err, [11, 14, 12], _f(F(2, 62), F(1, 65) + F(1, 61), F(1, 63) + F(1, 64)),
                                     60, 3)
    assert exact.ok and exact.n_subst == 2, exact.problems
    # 12 above 13 (fp32 may round either way): 12 = 2/63
    other = accept.check_dense_first(cand, lex, err, [11, 14, 12], _f(F(2, 62), F(1, 65) + F(1, 61), F(2, 63)), 60, 3)
    assert other.ok, other.problems
    # everything, with padding past the five candidates
    ids, vals = rrf.fuse_one((cand, [14, 11, 13, 12]), 60, 7)
    rep = accept.check_dense_first(cand, lex, err, ids, [rrf.to_f32(v) for v in vals], 60, 7)
    assert rep.ok, rep.problems


@pytest.mark.parametrize("ids,vals,why", [
    ([10, 11, 12], [Fraction(1, 61), Fraction(1, 62), Fraction(1, 63)], "dense order, no lexical rerank"),
    ([11, 14, 12], [Fraction(2, 62), Fraction(1, 65) + Fraction(1, 62), Fraction(2, 63)], "14 given lexical rank 2"),
    ([11, 12, 13], [Fraction(2, 62), Fraction(2, 63), Fraction(1, 64) + Fraction(1, 63)], "14 missed"),
    ([14, 11, 12], [Fraction(1, 65) + Fraction(1, 61), Fraction(2, 62), Fraction(2, 63)], "unordered"),
    ([11, 14, 10], [Fraction(2, 62), Fraction(1, 65) + Fraction(1, 61), Fraction(1, 61)], "10 before 12"),
    ([11, 14, 99], [Fraction(2, 62), Fraction(1, 65) + Fraction(1, 61), Fraction(1, 63)], "not a candidate"),
])
def test_dense_first_rejects_planted_mistakes(ids, vals, why):
    cand, lex, err = _df_case()
    rep = accept.check_dense_first(cand, lex, err, ids, _f(*vals), 60, 3)
    assert not rep.ok, why


def test_dense_first_completeness_uses_a_consistent_rank_order():
    """Candidates 2 and 3 are lexically near-tied (ranks 1 and 2 either way).  Returning 3 at
    lexical rank 1 is admissible even though 2 at rank 1 would beat it: 2 then has rank 2.
    Claiming rank 2 for 3 forces rank 1 on 2, whose fused value then beats 3's."""
    cand = [1, 2, 3]
    lex = np.array([0.0, 5.0, 5.0 + 1e-9])
    err = accept.bm25_f32_err(lex, 8)
    F = Fraction
    assert accept.check_dense_first(cand, lex, err, [3], _f(F(1, 63) + F(1, 61)), 60, 1).ok
    assert accept.check_dense_first(cand, lex, err, [2], _f(F(1, 62) + F(1, 61)), 60, 1).ok
    rep = accept.check_dense_first(cand, lex, err, [3], _f(F(1, 63) + F(1, 62)), 60, 1)
    assert not rep.ok
    # the order existence on its own: a chain with a fixed middle and a late release
    above = lambda x, y: x < y
    assert accept._rank_order_exists([0, 1, 2], above, {1: 2}, {2: 3})
    assert not accept._rank_order_exists([0, 1, 2], above, {1: 1}, {})
    assert not accept._rank_order_exists([0, 1, 2], lambda x, y: False, {0: 1}, {1: 3, 2: 3})


def test_dense_first_equal_signatures_fix_the_id_order():
    """Equal scores from equal (term, tf, length) contributions are computed bit-identically,
    so only the id order is admissible between them; without the signatures either is."""
    cand, lex = [20, 21], np.array([2.0, 2.0])
    err = accept.bm25_f32_err(lex, 8)
    right = _f(Fraction(2, 61), Fraction(2, 62))
    swapped = _f(Fraction(1, 61) + Fraction(1, 62), Fraction(1, 62) + Fraction(1, 61))
    assert accept.check_dense_first(cand, lex, err, [20, 21], right, 60, 2, sig=["a", "a"]).ok
    assert not accept.check_dense_first(cand, lex, err, [20, 21], swapped, 60, 2, sig=["a", "a"]).ok
    assert accept.check_dense_first(cand, lex, err, [20, 21], swapped, 60, 2, sig=["a", "b"]).ok


@settings(max_examples=200, deadline=None)
@given(st.lists(st.floats(0.05, 30.0), min_size=1, max_size=8), st.lists(st.integers(1, 3), min_size=8, max_size=8),
       st.lists(st.floats(0.01, 1.0), min_size=8, max_size=8))
def test_bm25_f32_bound_covers_fp32_sums(idf, mult, w):
    """bm25_f32_err bounds fp32 evaluations of a BM25 sum: factors rounded to fp32, products
    and additions rounded to fp32 one by one, in query order."""
    n = len(idf)
    exact = sum(i * m * x for i, m, x in zip(idf, mult, w))
    acc = np.float32(0.0)
    for i, m, x in zip(idf, mult, w):
        acc = np.float32(acc + np.float32(np.float32(np.float32(i) * np.float32(m)) * np.float32(x)))
    assert abs(float(acc) - exact) <= accept.bm25_f32_err(np.array([exact]), n)[0]


def test_gamma():
    assert accept.gamma(1024) == pytest.approx(1024 * 2 ** -23 / (1 - 1024 * 2 ** -23))
