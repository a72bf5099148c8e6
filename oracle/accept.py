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


def certificate(s_returned: np.ndarray, gpu_ids, gpu_scores, err_returned: np.ndarray, k: int, n_rows: int,
                s_unreturned=None, err_unreturned=None) -> Report:
    """Sort-free check for one query at full size.

    ``s_returned`` [k] are the oracle scores of the returned ids (any value in padding slots)
    and ``err_returned`` their error bounds.  The list must hold exactly min(k, n_rows)
    distinct ids in [0, n_rows) followed by -1 padding with -inf scores, match the oracle
    scores within the bounds, and be ordered.  ``s_unreturned`` / ``err_unreturned`` give
    oracle scores and bounds of rows NOT returned (every row that could matter: at least
    those scoring above the k-th returned score plus its bound); none of them may beat the
    k-th returned row by more than the two bounds.
    """
    rep = Report()
    g = np.asarray(gpu_ids, dtype=np.int64).reshape(-1)
    sh = np.asarray(gpu_scores, dtype=np.float64).reshape(-1)
    s_returned = np.asarray(s_returned, dtype=np.float64).reshape(-1)
    err_returned = np.asarray(err_returned, dtype=np.float64).reshape(-1)
    kk = min(k, n_rows)
    if g.shape[0] != k:
        rep.fail(f"list has {g.shape[0]} slots, expected {k}")
        return rep
    if np.any(g[:kk] < 0) or np.any(g[:kk] >= n_rows) or len(set(g[:kk].tolist())) != kk:
        rep.fail(f"ids are not {kk} distinct rows of [0, {n_rows}): {g[:kk].tolist()}")
        return rep
    if np.any(g[kk:] != -1) or np.any(np.isfinite(sh[kk:])):
        rep.fail(f"padding past {kk} entries is not (-1, -inf): {g[kk:].tolist()}")
        return rep
    for r in range(kk):
        if not abs(sh[r] - s_returned[r]) <= err_returned[r]:
            rep.fail(f"score parity r={r}: gpu {sh[r]!r} oracle {s_returned[r]!r}")
    for r in range(kk - 1):
        if sh[r] < sh[r + 1] or (sh[r] == sh[r + 1] and g[r] > g[r + 1]):
            rep.fail(f"gpu list not ordered at r={r}")
    if s_unreturned is not None and kk:
        s_u = np.asarray(s_unreturned, dtype=np.float64).reshape(-1)
        e_u = np.zeros_like(s_u) if err_unreturned is None else np.asarray(err_unreturned, dtype=np.float64).reshape(-1)
        j = int(np.argmin(s_returned[:kk]))
        kth = float(s_returned[j])
        beat = s_u > kth + err_returned[j] + e_u
        if np.any(beat):
            rep.fail(f"missed {int(beat.sum())} row(s), best scoring {float(s_u[beat].max())!r}, "
                     f"above the k-th returned {kth!r}")
    return rep


def bm25_f32_err(B: np.ndarray, n_terms) -> np.ndarray:
    """Bound on |fp32 BM25 - B| for a sum of positive contributions over at most ``n_terms``
    query terms.  Each contribution's factors are rounded to fp32 three times (idf (k1 + 1),
    the query multiplicity, the posting weight) and each of the at most n_terms additions
    rounds once, all relative errors of at most u = 2^-24 on positive values, so the sum is
    within gamma_{n_terms + 3}(u) B; the factor 2 absorbs the fp64 rounding of the attach-time
    factors."""
    n = np.asarray(n_terms, dtype=np.float64)
    u = 2.0 ** -24
    return 2.0 * (n + 3) * u / (1.0 - (n + 3) * u) * np.abs(np.asarray(B, dtype=np.float64))


def _rank_order_exists(items, above, fixed, release) -> bool:
    """Is there a bijection rank: items -> 1..n with rank[x] < rank[y] whenever above(x, y),
    rank[x] == fixed[x] where given and rank[x] >= release[x] where given?

    Unit jobs on one machine with precedence, release times and deadlines (a fixed rank is a
    release and a deadline at once, every other job may finish by n): release times are
    pushed forward and deadlines backward along the precedence relation, then the slots are
    filled in order by earliest modified deadline among the released jobs whose predecessors
    are placed.  For unit jobs with integer release times this rule finds a schedule whenever
    one exists (Lageweg, Lenstra and Rinnooy Kan, 1976), and here every slot must be used."""
    items = list(items)
    n = len(items)
    preds = {y: [x for x in items if x != y and above(x, y)] for y in items}
    succs = {x: [y for y in items if y != x and above(x, y)] for x in items}
    r = {x: fixed.get(x, release.get(x, 1)) for x in items}
    d = {x: fixed.get(x, n) for x in items}
    # the relation is a strict order (transitive), so one pass in a linear extension suffices
    topo = sorted(items, key=lambda x: len(preds[x]))
    for y in topo:
        for x in preds[y]:
            r[y] = max(r[y], r[x] + 1)
    for x in reversed(topo):
        for y in succs[x]:
            d[x] = min(d[x], d[y] - 1)
    if any(r[x] > d[x] for x in items):
        return False
    placed = set()
    for t in range(1, n + 1):
        ready = [x for x in items if x not in placed and r[x] <= t and all(p in placed for p in preds[x])]
        if not ready:
            return False
        x = min(ready, key=lambda z: (d[z], z))
        if d[x] < t:
            return False
        placed.add(x)
    return True


def check_dense_first(cand_ids, lex, lex_err, gpu_ids, gpu_fused, rrf_k: int, k: int, sig=None) -> Report:
    """Tie-aware check of a dense-first fused list for one query.

    ``cand_ids`` are the dense candidates in dense order (-1 = empty slot), ``lex`` their
    fp64 oracle lexical scores, ``lex_err`` bounds on the computed (fp32) scores' errors, and
    ``sig`` (optional) one hashable per candidate such that equal signatures guarantee
    bitwise equal computed scores (then only the id order is admissible between them).

    The lexical rank of a candidate with a positive score is known only up to the
    candidates whose scores lie within the two bounds of its own: its admissible ranks run
    from 1 + (candidates certainly above) to 1 + (candidates possibly above).  Accepted iff
      * the list holds min(k, candidates) distinct candidates, then (-1, -inf) padding;
      * each returned fused value is exactly fp32(1/(rrf_k + a) + 1/(rrf_k + r)) for the
        id's dense rank a and an admissible lexical rank r (1/(rrf_k + a) alone for a
        candidate without a positive score), and the recovered ranks are distinct;
      * the list is ordered by (exact fused value desc, id asc);
      * some admissible lexical order (ranks consistent with the candidates certainly above
        one another, the returned candidates at their recovered ranks) leaves every candidate
        that is not returned behind the k-th returned entry in (fused desc, id asc).
    Without near ties every interval is a single rank, and this is exact equality with the
    reranking of the candidates by their exact scores.
    """
    from fractions import Fraction

    rep = Report()
    cand = [int(c) for c in cand_ids]
    valid = [c for c in cand if c >= 0]
    a_of = {c: i + 1 for i, c in enumerate(valid)}
    lex_of = {c: float(v) for c, v in zip(cand, lex) if c >= 0}
    err_of = {c: float(e) for c, e in zip(cand, lex_err) if c >= 0}
    sig_of = {c: s for c, s in zip(cand, sig)} if sig is not None else {}
    pos = [c for c in valid if lex_of[c] > 0]

    def certainly_above(x, y):  # x's computed score beats y's, whatever the rounding
        if sig_of and sig_of.get(x) == sig_of.get(y) and lex_of[x] == lex_of[y]:
            return x < y
        return lex_of[x] - err_of[x] > lex_of[y] + err_of[y]

    rmin, rmax = {}, {}
    for c in pos:
        above = sum(1 for o in pos if o != c and certainly_above(o, c))
        below = sum(1 for o in pos if o != c and certainly_above(c, o))
        rmin[c], rmax[c] = 1 + above, len(pos) - below

    def dense_part(c):
        return Fraction(1, rrf_k + a_of[c])

    g = [int(x) for x in np.asarray(gpu_ids).reshape(-1)]
    f = np.asarray(gpu_fused, dtype=np.float32).reshape(-1)
    kk = min(k, len(valid))
    if len(g) != k or any(x < 0 for x in g[:kk]) or any(x != -1 for x in g[kk:]):
        rep.fail(f"expected {kk} ids then -1 padding: {g}")
        return rep
    if np.any(np.isfinite(f[kk:])):
        rep.fail("padding slots carry finite fused values")
    got = g[:kk]
    if len(set(got)) != kk or any(x not in a_of for x in got):
        rep.fail(f"ids repeated or not candidates: {got}")
        return rep
    exact, ranks = [], []
    for r, c in enumerate(got):
        if c in rmin:
            hit = None
            for lr in range(rmin[c], rmax[c] + 1):
                v = dense_part(c) + Fraction(1, rrf_k + lr)
                if np.float32(float(v)) == f[r]:
                    hit = (v, lr)
                    break
            if hit is None:
                rep.fail(f"slot {r}: id {c} (dense rank {a_of[c]}, lexical ranks {rmin[c]}..{rmax[c]}) "
                         f"has fused {f[r]!r}, no admissible value")
                return rep
            exact.append(hit[0])
            ranks.append(hit[1])
        else:
            v = dense_part(c)
            if np.float32(float(v)) != f[r]:
                rep.fail(f"slot {r}: id {c} has no lexical score, fused {f[r]!r} != 1/({rrf_k}+{a_of[c]})")
                return rep
            exact.append(v)
    if len(set(ranks)) != len(ranks):
        rep.fail(f"two returned candidates share a lexical rank: {ranks}")
    for r in range(kk - 1):
        if exact[r] < exact[r + 1] or (exact[r] == exact[r + 1] and got[r] > got[r + 1]):
            rep.fail(f"list not ordered at slot {r}")
    if kk:
        # Completeness: some admissible lexical order must put every candidate left out behind
        # the k-th returned entry.  The returned candidates keep their recovered ranks; a
        # candidate c left out needs a rank of at least m_c (the first at which its fused value
        # loses to the k-th); ranks are a permutation of 1..|positive| consistent with the
        # "certainly above" relations.
        fk, ik = exact[-1], got[-1]

        def loses(v, c):
            return v < fk or (v == fk and c > ik)

        fixed = {c: lr for c, lr in zip([c for c in got if c in rmin], ranks)}
        release = {}
        for c in valid:
            if c in got:
                continue
            if c not in rmin:
                if not loses(dense_part(c), c):
                    rep.fail(f"candidate {c} without a lexical score (fused {float(dense_part(c))!r}) beats the "
                             f"k-th returned {ik} ({float(fk)!r})")
                    return rep
                continue
            m = next((lr for lr in range(1, len(pos) + 1) if loses(dense_part(c) + Fraction(1, rrf_k + lr), c)), None)
            if m is None:
                rep.fail(f"candidate {c} beats the k-th returned {ik} at every lexical rank")
                return rep
            release[c] = m
        if not _rank_order_exists(pos, certainly_above, fixed, release):
            rep.fail(f"no admissible lexical order leaves the unreturned candidates behind the k-th returned {ik} "
                     f"({float(fk)!r}) with the returned ranks {dict(fixed)}")
    rep.n_subst = sum(1 for c in pos if rmax[c] > rmin[c])  # candidates with an uncertain rank
    return rep
