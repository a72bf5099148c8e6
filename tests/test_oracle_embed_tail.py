"""Pins for the embedding-tail oracle (mean pool + L2 normalisation): hand cases
(tests/golden/embed_tail_hand.yaml) and properties fixed by the definition: unit norm,
indifference to padding contents and to the order and common positive scale of the valid
tokens, and one valid token giving that token's direction."""
import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import embed_tail


def test_hand_cases(load_golden):
    for c in load_golden("embed_tail_hand.yaml")["cases"]:
        H = np.array([c["hidden"]], dtype=np.float64)
        out = embed_tail.pool(H, [c["len"]])[0]
        np.testing.assert_allclose(out, c["out"], rtol=0, atol=1e-14)


@settings(max_examples=80, deadline=None)
@given(st.integers(0, 10**6), st.integers(1, 9), st.floats(0.01, 100.0))
def test_properties(seed, n, scale):
    g = np.random.default_rng(seed)
    T, h = 9, 6
    H = g.normal(size=(1, T, h))
    out = embed_tail.pool(H, [n])[0]
    assert abs(np.linalg.norm(out) - 1) < 1e-12
    H2 = H.copy()
    H2[0, n:] = g.normal(size=(T - n, h)) * 1e3            # padding is ignored
    assert np.allclose(embed_tail.pool(H2, [n])[0], out, atol=1e-12)
    P = H.copy()
    P[0, :n] = H[0, g.permutation(n)]                        # token order is ignored
    assert np.allclose(embed_tail.pool(P, [n])[0], out, atol=1e-12)
    assert np.allclose(embed_tail.pool(scale * H, [n])[0], out, atol=1e-12)
    one = embed_tail.pool(H, [1])[0]
    assert np.allclose(one, H[0, 0] / np.linalg.norm(H[0, 0]), atol=1e-12)


def test_planted_mistake_fails(load_golden):
    """Averaging over every token (padding included) changes the first hand case."""
    c = load_golden("embed_tail_hand.yaml")["cases"][0]
    H = np.array(c["hidden"], dtype=np.float64)
    wrong = H.mean(axis=0) / np.linalg.norm(H.mean(axis=0))
    assert not np.allclose(wrong, c["out"], atol=1e-6)
