"""Tie-aware acceptance of a GPU ranked list against oracle scores.  Test infrastructure only.

The GPU accumulates in fp32 while the oracle scores in fp64, so two rows whose oracle
scores are closer than the GPU's rounding error may legitimately trade places.  A GPU list
(g, s_hat) for one query is accepted iff, with s the oracle scores, o the oracle's top-k
and near(a, b) the near-tie relation of the chosen mode:

  (i)   ids are distinct, valid (ranked by the oracle), and the list has exactly as many
        entries as the oracle's (the rest padded with -1);
  (ii)  |s_hat_r - s[g_r]| <= err[g_r] for every r                     (score parity);
  (iii) near(g_r, o_r) or g_r == o_r for every r                        (substitution only
        inside a near-tie run, including across the k-th boundary);
  (iv)  g_r == o_r wherever o_r is near-tied to no other ranked row;
  (v)   the GPU list is itself ordered: s_hat non-increasing, equal s_hat by ascending id.

Modes:
  ``rel``    - err = rtol * max(|s|, 1e-2); near(a, b) iff |s_a - s_b| < rtol * max(|s_a|, |s_b|, 1e-2).
               rtol = 2e-3 for bf16 / fp16 inputs, 1e-5 for fp32 inputs and for BM25.
  ``strict`` - err = per-row rigorous bound of an fp32 sum of exact products,
               2 * gamma_d * sum_j |q_j x_j|, gamma_d = d u / (1 - d u), u = 2^-23 (covers
               truncating as well as round-to-nearest accumulation); near(a, b) iff
               |s_a - s_b| <= err_a + err_b.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

FLOOR = 1e-2


def gamma(d: int, u: float = 2.0 ** -23) -> float:
    return d * u / (1.0 - d * u)


def strict_err(absdot: np.ndarray, d: int) -> np.ndarray:
    return 2.0 * gamma(d) * np.asarray(absdot, dtype=np.float64)


def rel_err(s: np.ndarray, rtol: float) -> np.ndarray:
    return rtol * np.maximum(np.abs(np.asarray(s, dtype=np.float64)), FLOOR)


@dataclass
class Report:
    ok: bool = True
    problems: list = field(default_factory=list)
    recall_raw: float = 1.0      # |g ∩ o| / |o|
    recall: float = 1.0          # near-tie substitutions counted as hits
    n_subst: int = 0

    def fail(self, msg: str) -> None:
        self.ok = False
        if len(self.problems) < 20:
            self.problems.append(msg)


def _near(mode, rtol, sa, sb, ea, eb):
    if mode == "strict":
        return abs(sa - sb) <= ea + eb
    return abs(sa - sb) < rtol * max(abs(sa), abs(sb), FLOOR)


def check_ranked(s: np.ndarray, gpu_ids, gpu_scores, k: int, *, mode: str = "rel", rtol: float = 2e-3,
                 err: np.ndarray | None = None, ranked: np.ndarray | None = None) -> Report:
    """Check one query's GPU list against the full oracle score vector ``s`` [N].

    ``ranked`` (bool [N]) marks the rows that take part in the ranking (all rows for dense
    search; chunks with a positive score for BM25).  ``err`` [N] is the per-row error bound
    (required for ``strict``; derived from ``rtol`` for ``rel``).
    """
    s = np.asarray(s, dtype=np.float64)
    n = s.shape[0]
    ranked = np.ones(n, dtype=bool) if ranked is None else np.asarray(ranked, dtype=bool)
    if err is None:
        if mode == "strict":
            raise ValueError("strict mode needs err")
        err = rel_err(s, rtol)
    err = np.asarray(err, dtype=np.float64)
    g = np.asarray(gpu_ids, dtype=np.int64).reshape(-1)
    sh = np.asarray(gpu_scores, dtype=np.float64).reshape(-1)
    rep = Report()

    pos = np.flatnonzero(ranked)
    order = pos[np.argsort(-s[pos], kind="stable")]
    kk = min(k, order.shape[0])
    o = order[:kk]

    # (i) validity and length
    nvalid = int(np.count_nonzero(g >= 0))
    if nvalid != kk or np.any(g[:kk] < 0) or np.any(g[kk:] != -1):
        rep.fail(f"list length {nvalid} (valid prefix) != expected {kk}: {g.tolist()}")
        return rep
    gv = g[:kk]
    if np.any(gv >= n) or len(set(gv.tolist())) != kk:
        rep.fail(f"ids out of range or repeated: {gv.tolist()}")
        return rep
    if not np.all(ranked[gv]):
        rep.fail(f"unranked ids returned: {gv[~ranked[gv]].tolist()}")
        return rep
    if np.any(np.isfinite(sh[kk:])):
        rep.fail("padding slots carry finite scores")

    # (ii) score parity
    for r in range(kk):
        i = gv[r]
        if not abs(sh[r] - s[i]) <= err[i]:
            rep.fail(f"score parity r={r} id={i}: gpu {sh[r]!r} oracle {s[i]!r} bound {err[i]:.3g}")

    # (v) the GPU's own order
    for r in range(kk - 1):
        if sh[r] < sh[r + 1] or (sh[r] == sh[r + 1] and gv[r] > gv[r + 1]):
            rep.fail(f"gpu list not ordered at r={r}: ({sh[r]!r},{gv[r]}) then ({sh[r+1]!r},{gv[r+1]})")

    # (iii) substitutions only between near-tied rows
    for r in range(kk):
        if gv[r] != o[r]:
            rep.n_subst += 1
            if not _near(mode, rtol, s[gv[r]], s[o[r]], err[gv[r]], err[o[r]]):
                rep.fail(f"rank {r}: gpu id {gv[r]} (s={s[gv[r]]!r}) for oracle id {o[r]} (s={s[o[r]]!r})")

    # (iv) isolated oracle rows must be exactly in place
    sorted_s = s[order]
    emax = float(err[order].max()) if order.shape[0] else 0.0
    for r in range(kk):
        i = o[r]
        wide = err[i] + emax + rtol * max(abs(s[i]), FLOOR) + 1e-300
        lo = np.searchsorted(-sorted_s, -(s[i] + wide), side="left")
        hi = np.searchsorted(-sorted_s, -(s[i] - wide), side="right")
        isolated = True
        for j in order[lo:hi]:
            if j != i and _near(mode, rtol, s[i], s[j], err[i], err[j]):
                isolated = False
                break
        if isolated and gv[r] != i:
            rep.fail(f"rank {r}: oracle id {i} is not near-tied to any row but gpu has {gv[r]}")

    inter = len(set(gv.tolist()) & set(o.tolist()))
    rep.recall_raw = inter / kk if kk else 1.0
    hits = 0
    oset = set(o.tolist())
    for r in range(kk):
        if gv[r] in oset or _near(mode, rtol, s[gv[r]], s[o[r]], err[gv[r]], err[o[r]]):
            hits += 1
    rep.recall = hits / kk if kk else 1.0
    return rep


def check_batch(S: np.ndarray, gpu_ids, gpu_scores, k: int, **kw):
    """check_ranked over a batch; ``err`` / ``ranked`` may be given per query as [B x N]."""
    err = kw.pop("err", None)
    ranked = kw.pop("ranked", None)
    reps = []
    for q in range(S.shape[0]):
        reps.append(check_ranked(S[q], gpu_ids[q], gpu_scores[q], k,
                                 err=None if err is None else err[q],
                                 ranked=None if ranked is None else ranked[q], **kw))
    return reps


def certificate(s_returned: np.ndarray, gpu_ids, gpu_scores, err_returned: np.ndarray,
                s_best_unreturned: float | None = None, err_best_unreturned: float = 0.0) -> Report:
    """Sort-free check for one query at full size.

    ``s_returned`` are the oracle scores of the returned ids.  When the oracle's best score
    among the rows NOT returned is given, nothing may beat the k-th returned row by more than
    the two error bounds.
    """
    rep = Report()
    g = np.asarray(gpu_ids, dtype=np.int64)
    sh = np.asarray(gpu_scores, dtype=np.float64)
    v = g >= 0
    kk = int(v.sum())
    if np.any(g[:kk] < 0) or len(set(g[:kk].tolist())) != kk:
        rep.fail("ids not a distinct valid prefix")
        return rep
    for r in range(kk):
        if not abs(sh[r] - s_returned[r]) <= err_returned[r]:
            rep.fail(f"score parity r={r}: gpu {sh[r]!r} oracle {s_returned[r]!r}")
    for r in range(kk - 1):
        if sh[r] < sh[r + 1] or (sh[r] == sh[r + 1] and g[r] > g[r + 1]):
            rep.fail(f"gpu list not ordered at r={r}")
    if s_best_unreturned is not None and kk:
        kth = float(np.min(s_returned[:kk]))
        j = int(np.argmin(s_returned[:kk]))
        if s_best_unreturned > kth + err_returned[j] + err_best_unreturned:
            rep.fail(f"missed a row scoring {s_best_unreturned!r} above the k-th returned {kth!r}")
    return rep
