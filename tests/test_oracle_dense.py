"""Pins for the dense oracle against hand values, exact integer arithmetic, a pure-Python
brute force and invariants of exact top-k (no GPU)."""
import math
import random

import numpy as np
import pytest

import synth
from oracle import dense as od
from oracle.storage import decode, round_f32_to_bf16, round_f32_to_f16


def test_hand_example(load_golden):
    g = load_golden("dense_hand.yaml")
    X = np.array(g["rows"], dtype=np.float64)
    q = np.array([g["query"]], dtype=np.float64)
    S = od.scores(X, q)
    np.testing.assert_allclose(S[0], g["scores"], rtol=0, atol=1e-15)
    ids, sc = od.topk_from_scores(S, 3)
    assert ids[0].tolist() == g["top3_ids"]
    s_self = od.scores(X, X[[g["self_query_row"]]])
    assert abs(s_self[0, g["self_query_row"]] - g["self_query_score"]) < 1e-15
    ids, _ = od.topk_from_scores(od.scores(X, np.array([g["tie_query"]])), 3)
    assert ids[0].tolist() == g["tie_top3_ids"]


def _py_topk(rows, q, k):
    """Independent formulation: exact rational dot products (Python ints / fractions of floats)
    and Python's sorted() on (-score, id)."""
    from fractions import Fraction
    sc = [sum(Fraction(a) * Fraction(b) for a, b in zip(q, r)) for r in rows]
    order = sorted(range(len(rows)), key=lambda i: (-sc[i], i))[:k]
    return order, [sc[i] for i in order]


def test_integer_vectors_exact_with_ties():
    rnd = np.random.default_rng(5)
    X = rnd.integers(-3, 4, size=(60, 7)).astype(np.float64)
    Q = rnd.integers(-3, 4, size=(9, 7)).astype(np.float64)
    ids, sc = od.topk_from_scores(od.scores(X, Q), 12)
    for b in range(Q.shape[0]):
        ref_ids, ref_sc = _py_topk(X.tolist(), Q[b].tolist(), 12)
        assert ids[b].tolist() == ref_ids
        assert [float(x) for x in ref_sc] == sc[b].tolist()


def test_bruteforce_float_rows():
    rnd = np.random.default_rng(11)
    X = rnd.standard_normal((64, 24))
    X /= np.linalg.norm(X, axis=1, keepdims=True)
    Q = rnd.standard_normal((5, 24))
    ids, sc = od.topk_from_scores(od.scores(X, Q), 10)
    for b in range(5):
        fs = [math.fsum(Q[b, j] * X[i, j] for j in range(24)) for i in range(64)]
        ref = sorted(range(64), key=lambda i: (-fs[i], i))[:10]
        assert ids[b].tolist() == ref
        np.testing.assert_allclose(sc[b], [fs[i] for i in ref], rtol=0, atol=1e-14)


def test_abs_dot_hand_case():
    """sum_j |q_j x_ij| by hand: row 0 -> 1 + 2 + 6 = 9, row 1 -> 0.5 + 0 + 8 = 8.5 (the plain
    dots are 3 and -8.5, so an absolute value taken after the sum fails row 0)."""
    X = np.array([[1.0, -2.0, 3.0], [0.5, 0.0, -4.0]])
    q = np.array([[-1.0, 1.0, 2.0], [0.0, 0.0, 0.0]])
    A = od.abs_dot(X, q)
    assert A.tolist() == [[9.0, 8.5], [0.0, 0.0]]
    assert od.scores(X, q)[0].tolist() == [3.0, -8.5]
    # never below |score|, equal for sign-consistent rows
    rnd = np.random.default_rng(8)
    Xr, Qr = rnd.standard_normal((30, 16)), rnd.standard_normal((4, 16))
    assert np.all(od.abs_dot(Xr, Qr) >= np.abs(od.scores(Xr, Qr)) - 1e-12)
    assert np.allclose(od.abs_dot(np.abs(Xr), np.abs(Qr)), od.scores(np.abs(Xr), np.abs(Qr)))


def test_padding_when_k_exceeds_rows():
    X = np.eye(3)
    ids, sc = od.topk_from_scores(od.scores(X, np.array([[0.1, 0.3, 0.2]])), 5)
    assert ids[0].tolist() == [1, 2, 0, -1, -1]
    assert np.isneginf(sc[0, 3:]).all()


def test_invariants_on_generated_workload():
    w = synth.tiny_dense()
    Xb = synth.storage_bits(w.rows)
    Qb = synth.storage_bits(w.queries)
    X = decode(Xb, "f32")
    # noise-free self-queries rank first
    self_ids, self_sc = od.topk_from_scores(od.scores(X, X[:40]), 1)
    assert self_ids[:, 0].tolist() == list(range(40))
    # prefix consistency, batch invariance
    i5, _ = od.topk(Xb, Qb, "f32", 5)
    i10, _ = od.topk(Xb, Qb, "f32", 10)
    assert (i10[:, :5] == i5).all()
    i5b, _ = od.topk(Xb, Qb[3:7], "f32", 5)
    assert (i5b == i5[3:7]).all()
    # permuting rows permutes ids (no ties in these draws)
    perm = np.random.default_rng(2).permutation(X.shape[0])
    ip, _ = od.topk(Xb[perm], Qb, "f32", 5)
    assert (perm[ip] == i5).all()
    # scores non-increasing and equal to recomputed dots
    _, s5 = od.topk(Xb, Qb, "f32", 5)
    assert (np.diff(s5, axis=1) <= 0).all()


def test_bf16_rounding_matches_torch_and_hand_cases():
    import torch
    rnd = np.random.default_rng(3)
    x = (rnd.standard_normal(20000) * 10.0 ** rnd.integers(-6, 6, 20000)).astype(np.float32)
    # exact halfway cases: low 16 bits = 0x8000, with even and odd upper halves
    half = (rnd.integers(0, 2 ** 15, 2000, dtype=np.uint32) << 16 | 0x8000).astype(np.uint32).view(np.float32)
    x = np.concatenate([x, half[np.isfinite(half)], np.array([0.0, -0.0, 1.0, -2.5, 65504.0], np.float32)])
    ours = round_f32_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (ours == ref).all()
    # hand cases: 1 + 2^-8 (bf16 ulp at 1 is 2^-7) is a tie -> rounds to even (1.0);
    # 1 + 3*2^-8 is a tie between 1+2^-7 (odd) and 1+2^-6 (even) -> 1 + 2^-6
    assert decode(round_f32_to_bf16(np.float32(1 + 2 ** -8)), "bf16") == 1.0
    assert decode(round_f32_to_bf16(np.float32(1 + 3 * 2 ** -8)), "bf16") == 1 + 2 ** -6
    h = round_f32_to_f16(np.float32(1 + 2 ** -11))
    assert decode(h, "f16") == 1.0


def test_decode_exact():
    assert decode(np.array([0x3F80], np.uint16), "bf16")[0] == 1.0
    assert decode(np.array([0xC000], np.uint16), "bf16")[0] == -2.0
    assert decode(np.array([0x3C00], np.uint16), "f16")[0] == 1.0
    assert decode(np.array([0x3F800000], np.uint32), "f32")[0] == 1.0


def test_self_query_rank_one_mixture():
    w = synth.mixture_dense(99, 4096, 256, 32, 8, 5, "bf16")
    X = decode(synth.storage_bits(w.rows), "bf16")
    ids, _ = od.topk_from_scores(od.scores(X, X[100:164]), 1)
    assert ids[:, 0].tolist() == list(range(100, 164))
