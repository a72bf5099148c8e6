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


def test_certificate():
    rep = accept.certificate(np.array([0.9, 0.8]), np.array([5, 2]), np.array([0.9, 0.8]), np.array([1e-6, 1e-6]),
                             s_best_unreturned=0.79)
    assert rep.ok
    rep = accept.certificate(np.array([0.9, 0.8]), np.array([5, 2]), np.array([0.9, 0.8]), np.array([1e-6, 1e-6]),
                             s_best_unreturned=0.85)
    assert not rep.ok


def test_gamma():
    assert accept.gamma(1024) == pytest.approx(1024 * 2 ** -23 / (1 - 1024 * 2 ** -23))
