"""BM25 over CSR postings, RRF fusion and the hybrid path on the GPU against the oracle."""
import numpy as np
import pytest
import torch

import synth
from oracle import accept, bm25, dense_first, rrf
from oracle import dense as od
from tests.gpu_helpers import check_dense, device, log, make_index, oracle_scores

pytestmark = pytest.mark.gpu


def _t(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def _attach(idx, csr, dev, k1=1.2, b=0.75):
    idx.attach_sparse(_t(csr.term_indptr, dev), _t(csr.post_chunk, dev), _t(csr.post_tf, dev),
                      _t(csr.doc_len, dev), k1, b)


def _check_sparse(B, ids, sc, k, label=""):
    ids = ids.cpu().numpy()
    sc = sc.cpu().numpy()
    bad = []
    for q in range(B.shape[0]):
        rep = accept.check_ranked(B[q], ids[q], sc[q], k, rtol=1e-5, ranked=B[q] > 0)
        if not rep.ok:
            bad.append((q, rep.problems))
    assert not bad, f"{label}: {len(bad)} queries fail, first {bad[:2]}"


def _small_corpus(seed, n_docs, vocab, mean_len, nq):
    ind, toks = synth.sparse_corpus(synth.rng(seed, 3), n_docs, vocab, 1.1, mean_len)
    csr = synth.csr_from_tokens(ind, toks, vocab)
    g = np.random.default_rng(seed)
    qs = [list(g.integers(0, vocab, size=g.integers(1, 9))) for _ in range(nq)]
    qs[0] = []                                 # no terms
    qs[1] = [-1, vocab, vocab + 5]             # only unknown terms
    qs[2] = [3, 3, 3, 0]                       # repeats
    qs[3] = [0, -7, 1]                         # known and unknown
    qi = np.zeros(nq + 1, dtype=np.int32)
    qi[1:] = np.cumsum([len(q) for q in qs])
    qt = np.array([t for q in qs for t in q], dtype=np.int32)
    return ind, toks, csr, qi, qt


@pytest.mark.parametrize("k", [1, 10, 100, 128])
def test_bm25_small_corpus(k):
    dev = device()
    ind, toks, csr, qi, qt = _small_corpus(500 + k, 3000, 400, 40.0, 60)
    idx = make_index(torch.zeros((3000, 128), dtype=torch.bfloat16), "bf16")
    _attach(idx, csr, dev)
    sc, ids = idx.search_sparse(_t(qi, dev), _t(qt, dev), k)
    torch.cuda.synchronize()
    qt_oracle = np.where((qt >= 0) & (qt < 400), qt, 10 ** 6).astype(np.int64)  # unknown terms match nothing
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    _check_sparse(B, ids, sc, k, f"k={k}")
    assert (ids.cpu()[0] == -1).all() and (ids.cpu()[1] == -1).all()


@pytest.mark.parametrize("k1,b", [(1.2, 0.75), (0.0, 0.75), (1.2, 0.0), (2.0, 1.0)])
def test_bm25_parameters(k1, b):
    dev = device()
    ind, toks, csr, qi, qt = _small_corpus(600, 2000, 300, 30.0, 40)
    idx = make_index(torch.zeros((2000, 128), dtype=torch.bfloat16), "bf16")
    _attach(idx, csr, dev, k1, b)
    sc, ids = idx.search_sparse(_t(qi, dev), _t(qt, dev), 50)
    torch.cuda.synchronize()
    qt_oracle = np.where((qt >= 0) & (qt < 300), qt, 10 ** 6).astype(np.int64)
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, k1, b)
    _check_sparse(B, ids, sc, 50, f"k1={k1} b={b}")


@pytest.mark.parametrize("n_docs,k", [(70_001, 64), (360_001, 100)])
def test_bm25_several_chunk_ranges(n_docs, k):
    """More chunks than one workgroup's LDS accumulator (32,768): per-range lists are merged
    (3 x 64 composites per query fit the LDS ranking merge; 11 x 100 take the queue merge)."""
    dev = device()
    ind, toks, csr, qi, qt = _small_corpus(700, n_docs, 2000, 20.0, 30)
    idx = make_index(torch.zeros((n_docs, 128), dtype=torch.bfloat16), "bf16")
    _attach(idx, csr, dev)
    sc, ids = idx.search_sparse(_t(qi, dev), _t(qt, dev), k)
    torch.cuda.synchronize()
    qt_oracle = np.where((qt >= 0) & (qt < 2000), qt, 10 ** 6).astype(np.int64)
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    _check_sparse(B, ids, sc, k, f"multi-range n_docs={n_docs}")


def _bm25_sweep_cases(n_cases=14, seed=2609):
    """Seeded (n_docs, vocab, mean_len, nq, k, max_terms) draws: one chunk to several 32,768-chunk
    ranges, vocabularies from all-head to flat, short to long queries, k below and above the
    corpus size."""
    r = np.random.default_rng(seed)
    sizes = [1, 7, 300, 5000, 32768, 32769, 45000]
    out = []
    for i in range(n_cases):
        n = sizes[i % len(sizes)]
        out.append((n, int(r.choice([6, 60, 3000])), float(r.choice([3.0, 20.0, 60.0])),
                    int(r.choice([1, 7, 64, 300])), int(r.choice([1, 7, 100, 128])), int(r.choice([4, 12, 48]))))
    return out


@pytest.mark.parametrize("n_docs,vocab,mean_len,nq,k,max_terms", _bm25_sweep_cases())
def test_bm25_seeded_sweep(n_docs, vocab, mean_len, nq, k, max_terms):
    """BM25 top-k over seeded corpora and query batches against the token-scan oracle
    (rtol 1e-5), including chunks with no positive score, queries without known terms and
    queries longer than one 32-occurrence parse batch."""
    log("bm25 sweep", n_docs, vocab, mean_len, nq, k, max_terms)
    dev = device()
    g = np.random.default_rng(n_docs + vocab + nq + k)
    ind, toks = synth.sparse_corpus(synth.rng(900 + n_docs % 97, 3), n_docs, vocab, 1.1, mean_len)
    csr = synth.csr_from_tokens(ind, toks, vocab)
    qs = [list(g.integers(-2, vocab + 2, size=g.integers(0, max_terms + 1))) for _ in range(nq)]
    qi = np.zeros(nq + 1, dtype=np.int32)
    qi[1:] = np.cumsum([len(q) for q in qs])
    qt = np.array([t for q in qs for t in q], dtype=np.int32)
    idx = make_index(torch.zeros((n_docs, 128), dtype=torch.bfloat16), "bf16")
    _attach(idx, csr, dev)
    sc, ids = idx.search_sparse(_t(qi, dev), _t(qt, dev), k)
    torch.cuda.synchronize()
    qt_oracle = np.where((qt >= 0) & (qt < vocab), qt, 10 ** 6).astype(np.int64)
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    _check_sparse(B, ids, sc, k, f"n_docs={n_docs} vocab={vocab} nq={nq} k={k}")


@pytest.mark.parametrize("kind", ["no_head", "one_head", "all_head"])
def test_bm25_head_rows_and_postings_mix(kind):
    """The most frequent terms (df >= N / 8) are scored from dense rows, the rest from their
    postings.  A flat corpus (uniform tokens, no term that frequent) takes only postings; one
    term in every chunk gives a single head row next to ordinary terms; a 12-term vocabulary
    makes every term a head term.  Queries mix kinds, repeat terms and include unknown ones;
    scores within rtol 1e-5 of the token-scan oracle, and dense-first (same summation order)
    scores its candidates identically to the full search (one query is longer than the
    32 occurrences dense-first holds at once)."""
    dev = device()
    g = np.random.default_rng({"no_head": 61, "one_head": 62, "all_head": 63}[kind])
    n, vocab = 3000, 2000 if kind != "all_head" else 12
    lens = g.integers(5, 40, size=n)
    docs = [list(g.integers(1 if kind == "one_head" else 0, vocab, size=m)) for m in lens]
    if kind == "one_head":
        docs = [d + [0] * int(g.integers(1, 4)) for d in docs]  # term 0 in every chunk
    ind = np.zeros(n + 1, dtype=np.int64)
    ind[1:] = np.cumsum([len(d) for d in docs])
    toks = np.array([t for d in docs for t in d], dtype=np.int32)
    csr = synth.csr_from_tokens(ind, toks, vocab)
    nq = 48
    qs = [list(g.integers(0, vocab, size=g.integers(1, 9))) for _ in range(nq)]
    qs[0] = [0, 0, 5, -1]
    qs[1] = [3, 0, 3]
    qs[2] = list(g.integers(0, vocab, size=45)) + [0, 1, 0]  # longer than one 32-term batch
    qi = np.zeros(nq + 1, dtype=np.int32)
    qi[1:] = np.cumsum([len(q) for q in qs])
    qt = np.array([t for q in qs for t in q], dtype=np.int32)
    w = synth.mixture_dense(6400 + len(kind), n, 128, 16, nq, 64, "bf16")
    idx = make_index(w.rows, "bf16")
    _attach(idx, csr, dev)
    log("bm25 head rows", kind)
    sc, ids = idx.search_sparse(_t(qi, dev), _t(qt, dev), 64)
    fused, fids = idx.search_hybrid_dense_first(w.queries.to(dev), _t(qi, dev), _t(qt, dev), 64, 60, 64)
    dsc, dids = idx.search_dense(w.queries.to(dev), 64)
    torch.cuda.synchronize()
    qt_oracle = np.where((qt >= 0) & (qt < vocab), qt, 10 ** 6).astype(np.int64)
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    _check_sparse(B, ids, sc, 64, kind)
    _check_dense_first(fused, fids, dids, B, qi, qt_oracle, ind, toks, 60, 64, f"dense-first {kind}")


def test_attach_rejects_malformed_csr():
    dev = device()
    from paper_2608_08340_amd import OpragError
    ind, toks, csr, qi, qt = _small_corpus(800, 500, 50, 10.0, 5)
    idx = make_index(torch.zeros((500, 128), dtype=torch.bfloat16), "bf16")
    bad = csr.post_chunk.copy()
    lo, hi = csr.term_indptr[0], csr.term_indptr[1]
    bad[lo], bad[lo + 1] = bad[lo + 1], bad[lo]            # not ascending within term 0
    with pytest.raises(OpragError):
        idx.attach_sparse(_t(csr.term_indptr, dev), _t(bad, dev), _t(csr.post_tf, dev), _t(csr.doc_len, dev))
    badtf = csr.post_tf.copy()
    badtf[5] = 0
    with pytest.raises(OpragError):
        idx.attach_sparse(_t(csr.term_indptr, dev), _t(csr.post_chunk, dev), _t(badtf, dev), _t(csr.doc_len, dev))
    with pytest.raises(OpragError):   # search before any successful attach
        idx.search_sparse(_t(qi, dev), _t(qt, dev), 5)


def test_rrf_kernel_matches_exact_fractions():
    dev = device()
    from paper_2608_08340_amd import rrf_fuse
    g = np.random.default_rng(9)
    nq, kd, ks = 200, 100, 100
    D = np.full((nq, kd), -1, np.int64)
    S = np.full((nq, ks), -1, np.int64)
    for q in range(nq):
        pool = g.permutation(300)
        nd, ns = int(g.integers(0, kd + 1)), int(g.integers(0, ks + 1))
        D[q, :nd] = pool[:nd]
        S[q, :ns] = g.permutation(pool[: max(ns, 1) + int(g.integers(0, 100))])[:ns]
    D[0], S[0] = -1, -1
    D[0, :3], S[0, :2] = [7, 3, 9], [3, 5]          # the hand example, lists otherwise empty
    for k in (5, 100, 128):
        fused, ids = rrf_fuse(_t(D, dev), _t(S, dev), 60, k)
        torch.cuda.synchronize()
        ref_ids, ref_f32, _ = rrf.fuse(D, S, 60, k)
        assert np.array_equal(ids.cpu().numpy(), ref_ids)
        assert np.array_equal(fused.cpu().numpy().view(np.uint32), ref_f32.view(np.uint32))
    # rrf_k across the kernel's two orderings: correctly rounded quotients (rrf_k < 1e5) and
    # quotients with exact int64 checks of near pairs (larger rrf_k)
    for rk in (0, 99_999, 100_000, 1_000_000):
        fused, ids = rrf_fuse(_t(D, dev), _t(S, dev), rk, 10)
        torch.cuda.synchronize()
        ref_ids, ref_f32, _ = rrf.fuse(D, S, rk, 10)
        assert np.array_equal(ids.cpu().numpy(), ref_ids), rk
        assert np.array_equal(fused.cpu().numpy().view(np.uint32), ref_f32.view(np.uint32)), rk


@pytest.fixture(scope="module")
def c3():
    device()
    return synth.hybrid_32k()


@pytest.mark.timeout(300)
@pytest.mark.parametrize("correlated", [False, True])
def test_hybrid_32k_bm25_rrf_top5(c3, correlated):
    """32,768 x 1,024 bf16 index + Zipf(1.1) CSR corpus (30,000 terms, Poisson(256) lengths),
    256 queries of 8 terms: dense top-100 and BM25 top-100 each pass the acceptance rules, and
    the fused top-5 equals exact RRF(60) of the GPU's own two lists."""
    dev = device()
    h = c3 if not correlated else synth.hybrid_32k(correlated=True, dense=synth.dense_32k())
    w = h.dense
    log("hybrid", "correlated" if correlated else "independent", tuple(w.rows.shape), h.csr.nnz)
    idx = make_index(w.rows, "bf16")
    _attach(idx, h.csr, dev, h.k1, h.b)
    q = w.queries.to(dev)
    qi, qt = _t(h.qterm_indptr, dev), _t(h.qterms, dev)
    fused, fids = idx.search_hybrid(q, qi, qt, 100, 100, 60, 5)
    dsc, dids = idx.search_dense(q, 100)
    ssc, sids = idx.search_sparse(qi, qt, 100)
    torch.cuda.synchronize()
    # stage 1: dense top-100
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    check_dense(S, X, Q, dids, dsc, 100, "bf16", label="dense top-100")
    # stage 2: BM25 top-100 from the raw token sequences
    B = bm25.scores_batch(h.doc_indptr, h.tokens, h.qterm_indptr, h.qterms, h.k1, h.b)
    _check_sparse(B, sids, ssc, 100, "bm25 top-100")
    # stage 3: exact RRF of the GPU's own lists, and equality with the composition
    ref_ids, ref_f32, _ = rrf.fuse(dids.cpu().numpy(), sids.cpu().numpy(), 60, 5)
    assert np.array_equal(fids.cpu().numpy(), ref_ids)
    assert np.array_equal(fused.cpu().numpy().view(np.uint32), ref_f32.view(np.uint32))
    # where the GPU lists equal the oracle lists, the fused output equals the oracle's
    od_ids, _ = od.topk_from_scores(S, 100)
    ob_ids, _ = bm25.sparse_topk_from_scores(B, 100)
    same = (dids.cpu().numpy() == od_ids).all(1) & (sids.cpu().numpy() == ob_ids).all(1)
    o_ids, _, _ = rrf.fuse(od_ids, ob_ids, 60, 5)
    assert same.mean() > 0.2
    assert np.array_equal(fids.cpu().numpy()[same], o_ids[same])
    log("queries whose stage lists equal the oracle's exactly:", int(same.sum()), "of", len(same))


OPRAG_MAX_K = 128


def _hybrid_sweep_cases(n_cases=10, seed=2610):
    """Seeded (n, d, nq, k_dense, k_sparse, rrf_k, k) draws for the RRF hybrid: corpora inside one
    32,768-chunk range (BM25 and RRF in one launch) and past it (separate RRF launch), fused k
    from 1 to the sum of both list lengths."""
    r = np.random.default_rng(seed)
    out = []
    for i in range(n_cases):
        n = [900, 5000, 32768, 40000][i % 4]
        kd, ks = int(r.choice([1, 5, 17, 100, 128])), int(r.choice([1, 5, 17, 100, 128]))
        k = int(min(kd + ks, OPRAG_MAX_K, r.choice([1, 5, 10, 64, 128])))
        out.append((n, int(r.choice([128, 384, 1024])), int(r.choice([1, 16, 100, 257])), kd, ks,
                    int(r.choice([0, 1, 60, 1000])), k))
    return out


@pytest.mark.timeout(300)
@pytest.mark.parametrize("n,d,nq,k_dense,k_sparse,rrf_k,k", _hybrid_sweep_cases())
def test_hybrid_seeded_sweep(n, d, nq, k_dense, k_sparse, rrf_k, k):
    """The one-call RRF hybrid over seeded shapes: its dense and BM25 stages pass the
    acceptance rules as stand-alone searches, and the fused list equals exact RRF of those two
    lists bit for bit."""
    log("hybrid sweep", n, d, nq, k_dense, k_sparse, rrf_k, k)
    dev = device()
    w = synth.mixture_dense(7000 + n % 101 + d, n, d, 32, nq, k_dense, "bf16")
    g = np.random.default_rng(n + nq)
    ind, toks = synth.sparse_corpus(synth.rng(950 + n % 89, 3), n, 2000, 1.1, 30.0)
    csr = synth.csr_from_tokens(ind, toks, 2000)
    qs = [list(g.integers(0, 2000, size=g.integers(0, 12))) for _ in range(nq)]
    qi = np.zeros(nq + 1, dtype=np.int32)
    qi[1:] = np.cumsum([len(q) for q in qs])
    qt = np.array([t for q in qs for t in q], dtype=np.int32)
    idx = make_index(w.rows, "bf16")
    _attach(idx, csr, dev)
    q = w.queries.to(dev)
    qit, qtt = _t(qi, dev), _t(qt, dev)
    fused, fids = idx.search_hybrid(q, qit, qtt, k_dense, k_sparse, rrf_k, k)
    dsc, dids = idx.search_dense(q, k_dense)
    ssc, sids = idx.search_sparse(qit, qtt, k_sparse)
    torch.cuda.synchronize()
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    check_dense(S, X, Q, dids, dsc, k_dense, "bf16", label="dense stage")
    B = bm25.scores_batch(ind, toks, qi, qt.astype(np.int64), 1.2, 0.75)
    _check_sparse(B, sids, ssc, k_sparse, "bm25 stage")
    ref_ids, ref_f32, _ = rrf.fuse(dids.cpu().numpy(), sids.cpu().numpy(), rrf_k, k)
    assert np.array_equal(fids.cpu().numpy(), ref_ids)
    assert np.array_equal(fused.cpu().numpy().view(np.uint32), ref_f32.view(np.uint32))


@pytest.mark.timeout(300)
def test_hybrid_other_stream_and_graph_replay(c3):
    """A hybrid search (threshold levels with device-side repair gates, BM25, RRF) issued on a
    non-default stream, and captured in a HIP graph replayed three times (outputs cleared and
    other searches run in between), equals the eager result bit for bit."""
    dev = device()
    h = c3
    w = h.dense
    idx = make_index(w.rows, "bf16")
    _attach(idx, h.csr, dev, h.k1, h.b)
    q = w.queries.to(dev)
    qi, qt = _t(h.qterm_indptr, dev), _t(h.qterms, dev)
    ref_f, ref_i = idx.search_hybrid(q, qi, qt, 100, 100, 60, 5)
    torch.cuda.synchronize()
    log("hybrid on another stream")
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s):
        f2, i2 = idx.search_hybrid(q, qi, qt, 100, 100, 60, 5)
    s.synchronize()
    assert torch.equal(i2, ref_i) and torch.equal(f2.view(torch.int32), ref_f.view(torch.int32))
    log("hybrid captured in a graph")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fg, ig = idx.search_hybrid(q, qi, qt, 100, 100, 60, 5)
    torch.cuda.synchronize()
    for rep in range(3):
        fg.fill_(-1.0)
        ig.fill_(-2)
        g.replay()
        idx.search_dense(q[:7], 5)  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(ig, ref_i), f"replay {rep}"
        assert torch.equal(fg.view(torch.int32), ref_f.view(torch.int32)), f"replay {rep}"


def _signatures(cand, lex, terms, doc_indptr, tokens):
    """One hashable per candidate; equal signatures mean equal (term, tf) matches and equal
    length, which the GPU turns into bit-identical scores.  Only candidates whose fp64 score
    equals another candidate's need a real one."""
    sig = [("unique", int(c)) for c in cand]
    vals, counts = np.unique(lex[lex > 0], return_counts=True)
    tied = set(vals[counts > 1].tolist())
    distinct = list(dict.fromkeys(int(t) for t in terms))
    for i, c in enumerate(cand):
        if c >= 0 and lex[i] in tied:
            toks = tokens[doc_indptr[c]:doc_indptr[c + 1]]
            sig[i] = (len(toks),) + tuple(int(np.count_nonzero(toks == t)) for t in distinct)
    return sig


def _check_dense_first(fused, fids, dids, B, qi, qt, doc_indptr, tokens, rrf_k, k, label):
    """Tie-aware check of every query (oracle.accept.check_dense_first): the lexical rank of
    each candidate is fixed up to the candidates whose fp64 BM25 scores lie within the fp32
    error bounds of its own, and every returned fused value must be the exact RRF value of an
    admissible rank; queries without such near ties are checked for exact equality with the
    oracle's reranking.  B [nq x N] holds the fp64 BM25 score of every chunk (0 past the
    sparse corpus)."""
    dids = dids.cpu().numpy()
    g_ids, g_f = fids.cpu().numpy(), fused.cpu().numpy()
    e_ids, e_f, _ = dense_first.batch(dids, B, rrf_k, k)
    n_loose = n_exact = 0
    for q in range(dids.shape[0]):
        c = dids[q]
        lex = np.array([B[q, i] if i >= 0 else 0.0 for i in c])
        terms = qt[qi[q]:qi[q + 1]]
        err = accept.bm25_f32_err(lex, max(1, len(terms)))
        sig = _signatures(c, lex, terms, doc_indptr, tokens)
        rep = accept.check_dense_first(c, lex, err, g_ids[q], g_f[q], rrf_k, k, sig=sig)
        assert rep.ok, (label, q, rep.problems)
        if rep.n_subst:
            n_loose += 1
        else:  # no uncertain rank: the oracle's reranking exactly
            assert np.array_equal(g_ids[q], e_ids[q]), (label, q)
            assert np.array_equal(g_f[q].view(np.uint32), e_f[q].view(np.uint32)), (label, q)
            n_exact += 1
    log(f"{label}: {n_exact} queries without near ties (exact), {n_loose} with admissible rank intervals")


@pytest.mark.parametrize("n_cand,k", [(128, 5), (37, 10), (8, 20)])
def test_dense_first_small_corpus(n_cand, k):
    """Dense-first hybrid on 3,000 chunks (d = 128, 400 terms): the GPU's dense top-n_cand
    candidates, reranked by their BM25 scores and fused with their dense order by RRF(60),
    equal the oracle's fusion of the same candidates with fp64 BM25, fraction for fraction.
    Queries 0-3 have no terms, only unknown terms, repeats, and a mix."""
    dev = device()
    n, nq = 3000, 60
    ind, toks, csr, qi, qt = _small_corpus(900 + n_cand, n, 400, 40.0, nq)
    w = synth.mixture_dense(950 + n_cand, n, 128, 16, nq, n_cand, "bf16")
    idx = make_index(w.rows, "bf16")
    _attach(idx, csr, dev)
    q = w.queries.to(dev)
    log("dense-first small", n_cand, k)
    fused, fids = idx.search_hybrid_dense_first(q, _t(qi, dev), _t(qt, dev), n_cand, 60, k)
    dsc, dids = idx.search_dense(q, n_cand)
    torch.cuda.synchronize()
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    check_dense(S, X, Q, dids, dsc, n_cand, "bf16", label="candidates")
    qt_oracle = np.where((qt >= 0) & (qt < 400), qt, 10 ** 6).astype(np.int64)
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    _check_dense_first(fused, fids, dids, B, qi, qt_oracle, ind, toks, 60, k, f"n_cand={n_cand} k={k}")
    # no lexical evidence: the dense order alone
    d0 = dids.cpu().numpy()[0]
    assert np.array_equal(fids.cpu().numpy()[0][: min(k, n_cand)], d0[: min(k, n_cand)])


def test_dense_first_fewer_rows_than_candidates():
    """50 chunks, 128 candidates asked, k = 60: the 50 valid candidates are fused and the rest
    of each row is padding (-1, -inf)."""
    dev = device()
    n, nq = 50, 12
    ind, toks, csr, qi, qt = _small_corpus(1300, n, 30, 8.0, nq)
    w = synth.mixture_dense(1301, n, 128, 4, nq, 16, "bf16")
    idx = make_index(w.rows, "bf16")
    _attach(idx, csr, dev)
    q = w.queries.to(dev)
    fused, fids = idx.search_hybrid_dense_first(q, _t(qi, dev), _t(qt, dev), 128, 60, 60)
    dsc, dids = idx.search_dense(q, 128)
    torch.cuda.synchronize()
    qt_oracle = np.where((qt >= 0) & (qt < 30), qt, 10 ** 6).astype(np.int64)
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    _check_dense_first(fused, fids, dids, B, qi, qt_oracle, ind, toks, 60, 60, "50 rows")
    assert (fids.cpu().numpy()[:, 50:] == -1).all()
    assert np.isneginf(fused.cpu().numpy()[:, 50:]).all()


@pytest.mark.parametrize("n_cand,k", [(128, 5), (64, 64)])
def test_dense_first_index_past_the_sparse_corpus(n_cand, k):
    """3,000 dense rows over a 2,500-chunk sparse corpus: candidates at or past chunk 2,500
    have no postings (lexical score 0, dense rank only), as in weighted fusion.  The kernel
    must not read the chunk-major list of a chunk the corpus does not hold."""
    dev = device()
    n, n_docs, nq = 3000, 2500, 48
    ind, toks, csr, qi, qt = _small_corpus(3100 + k, n_docs, 300, 30.0, nq)
    w = synth.mixture_dense(3101 + k, n, 128, 16, nq, n_cand, "bf16")
    # half the queries are copies of rows past the corpus, so their candidates mix both kinds
    q32 = w.queries.float().numpy()
    rows32 = w.rows.float().numpy()
    q32[::2] = rows32[n_docs + 7 * np.arange(0, nq, 2) % (n - n_docs)]
    queries = synth.to_storage(q32, "bf16")
    idx = make_index(w.rows, "bf16")
    _attach(idx, csr, dev)
    log("dense-first past the corpus", n_cand, k)
    fused, fids = idx.search_hybrid_dense_first(queries.to(dev), _t(qi, dev), _t(qt, dev), n_cand, 60, k)
    dsc, dids = idx.search_dense(queries.to(dev), n_cand)
    torch.cuda.synchronize()
    d_np = dids.cpu().numpy()
    assert (d_np >= n_docs).any() and ((d_np >= 0) & (d_np < n_docs)).any()
    qt_oracle = np.where((qt >= 0) & (qt < 300), qt, 10 ** 6).astype(np.int64)
    B = np.zeros((nq, n))
    B[:, :n_docs] = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    _check_dense_first(fused, fids, dids, B, qi, qt_oracle, ind, toks, 60, k, f"past corpus n_cand={n_cand}")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("correlated", [False, True])
def test_dense_first_32k_against_oracle_and_full_hybrid(c3, correlated):
    """The 32,768 x 1,024 bf16 hybrid workload, 256 queries of 8 terms: dense-first with 128
    candidates and k = 5 matches the oracle's fusion of the GPU's candidates; Recall@5 and
    Jaccard overlap against full hybrid retrieval (RRF of dense and BM25 top-100 lists over
    the whole corpus) are logged, as the paper reports them.  They depend on how far the
    lexical and dense signals agree: little with independent synthetic queries, more when the
    query terms are drawn from the chunk the dense query was made from."""
    dev = device()
    h = c3 if not correlated else synth.hybrid_32k(correlated=True, dense=synth.dense_32k())
    w = h.dense
    idx = make_index(w.rows, "bf16")
    _attach(idx, h.csr, dev, h.k1, h.b)
    q = w.queries.to(dev)
    qi, qt = _t(h.qterm_indptr, dev), _t(h.qterms, dev)
    fused, fids = idx.search_hybrid_dense_first(q, qi, qt, 128, 60, 5)
    dsc, dids = idx.search_dense(q, 128)
    full_f, full_ids = idx.search_hybrid(q, qi, qt, 100, 100, 60, 5)
    torch.cuda.synchronize()
    B = bm25.scores_batch(h.doc_indptr, h.tokens, h.qterm_indptr, h.qterms, h.k1, h.b)
    _check_dense_first(fused, fids, dids, B, h.qterm_indptr, h.qterms, h.doc_indptr, h.tokens, 60, 5, "32k")
    a, b = fids.cpu().numpy(), full_ids.cpu().numpy()
    recall = np.mean([len(set(a[i]) & set(b[i])) / 5 for i in range(len(a))])
    jacc = np.mean([len(set(a[i]) & set(b[i])) / len(set(a[i]) | set(b[i])) for i in range(len(a))])
    log(f"dense-first vs full hybrid ({'correlated' if correlated else 'independent'} terms): "
        f"Recall@5 {recall:.3f}, Jaccard {jacc:.3f}")
    assert 0.0 <= jacc <= recall <= 1.0


def _check_weighted(F, sc, ids, k, label):
    reps = accept.check_batch(F, ids.cpu().numpy(), sc.cpu().numpy(), k, rtol=1e-3)
    bad = [(q, r.problems) for q, r in enumerate(reps) if not r.ok]
    assert not bad, f"{label}: {len(bad)} queries fail, first {bad[:2]}"


@pytest.mark.parametrize("w_d,w_l,k,n,n_docs,vocab", [(0.5, 0.5, 5, 3000, 2500, 300), (0.8, 0.2, 17, 3000, 2500, 300),
                                                     (1.0, 0.0, 10, 3000, 2500, 300), (0.0, 1.0, 10, 3000, 2500, 300),
                                                     (0.3, 0.7, 128, 3000, 2500, 300), (0.5, 0.5, 100, 70, 50, 300),
                                                     (0.5, 0.5, 5, 3000, 3000, 8)])
def test_weighted_fusion_small_corpus(w_d, w_l, k, n, n_docs, vocab):
    """Weighted fusion (min-max normalised dense and BM25 over every chunk) on a d = 128 index
    whose sparse corpus covers its first n_docs chunks (the rest score 0 lexically): the GPU
    top-k passes the acceptance rules against the fp64 oracle's fused scores.  Queries 0-3
    have no terms, only unknown terms, repeats and a mix (with w_l = 1 and no terms every
    chunk ties at 0).  k = 128 is the largest k; one case has fewer chunks than k; in the last
    the corpus covers every chunk with an 8-term vocabulary, so most queries have a lexical
    minimum above 0 (which padding past the last chunk must not lower)."""
    from oracle import weighted
    dev = device()
    nq = 40
    ind, toks, csr, qi, qt = _small_corpus(1500 + k, n_docs, vocab, 30.0, nq)
    w = synth.mixture_dense(1501 + k, n, 128, 16, nq, k, "bf16")
    idx = make_index(w.rows, "bf16")
    _attach(idx, csr, dev)
    log("weighted small", w_d, w_l, k, n, vocab)
    sc, ids = idx.search_hybrid_weighted(w.queries.to(dev), _t(qi, dev), _t(qt, dev), w_d, w_l, k)
    torch.cuda.synchronize()
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    qt_oracle = np.where((qt >= 0) & (qt < vocab), qt, 10 ** 6).astype(np.int64)
    B = np.zeros((nq, n))
    B[:, :n_docs] = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    _check_weighted(weighted.fused(S, B, w_d, w_l), sc, ids, k, f"w=({w_d},{w_l}) k={k}")


def _fusion_sweep_cases(n_cases=10, seed=2611):
    """Seeded (n, n_docs, d, nq, n_cand, k, w_dense, w_lex) draws for dense-first and weighted
    fusion: sparse corpora covering all or part of the index, one or several chunk ranges."""
    r = np.random.default_rng(seed)
    out = []
    for i in range(n_cases):
        n = [600, 4000, 32768, 40000][i % 4]
        n_docs = n if i % 3 else int(n * 0.8)
        w_d = float(r.choice([0.0, 0.25, 0.5, 1.0]))
        out.append((n, n_docs, int(r.choice([128, 384, 1024])), int(r.choice([1, 16, 100, 257])),
                    int(r.choice([1, 8, 64, 128])), int(r.choice([1, 5, 33, 128])), w_d, 1.0 - w_d))
    return out


@pytest.mark.timeout(300)
@pytest.mark.parametrize("n,n_docs,d,nq,n_cand,k,w_d,w_l", _fusion_sweep_cases())
def test_dense_first_and_weighted_seeded_sweep(n, n_docs, d, nq, n_cand, k, w_d, w_l):
    """Dense-first (tie-aware check against the oracle's reranking of the GPU's candidates)
    and weighted fusion (acceptance rules against the fp64 fused scores) over seeded shapes."""
    from oracle import weighted
    log("fusion sweep", n, n_docs, d, nq, n_cand, k, w_d, w_l)
    dev = device()
    w = synth.mixture_dense(7100 + n % 103 + d, n, d, 32, nq, n_cand, "bf16")
    g = np.random.default_rng(n + nq + k)
    ind, toks = synth.sparse_corpus(synth.rng(970 + n % 83, 3), n_docs, 1500, 1.1, 25.0)
    csr = synth.csr_from_tokens(ind, toks, 1500)
    qs = [list(g.integers(-1, 1501, size=g.integers(0, 40))) for _ in range(nq)]
    qi = np.zeros(nq + 1, dtype=np.int32)
    qi[1:] = np.cumsum([len(q) for q in qs])
    qt = np.array([t for q in qs for t in q], dtype=np.int32)
    idx = make_index(w.rows, "bf16")
    _attach(idx, csr, dev)
    q = w.queries.to(dev)
    qit, qtt = _t(qi, dev), _t(qt, dev)
    fused, fids = idx.search_hybrid_dense_first(q, qit, qtt, n_cand, 60, k)
    dsc, dids = idx.search_dense(q, n_cand)
    wsc, wids = idx.search_hybrid_weighted(q, qit, qtt, w_d, w_l, k)
    torch.cuda.synchronize()
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    check_dense(S, X, Q, dids, dsc, n_cand, "bf16", label="candidates")
    qt_oracle = np.where((qt >= 0) & (qt < 1500), qt, 10 ** 6).astype(np.int64)
    B = np.zeros((nq, n))
    B[:, :n_docs] = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    _check_dense_first(fused, fids, dids, B, qi, qt_oracle, ind, toks, 60, k, f"dense-first n={n} nq={nq}")
    _check_weighted(weighted.fused(S, B, w_d, w_l), wsc, wids, k, f"weighted n={n} w=({w_d},{w_l}) k={k}")


def test_weighted_fusion_index_smaller_than_its_corpus():
    """An index of 2,000 rows (capacity 3,000) over a 3,000-chunk sparse corpus, both inside
    one 32,768-chunk range: the fusion covers the chunks with a dense row only, so the lexical
    minimum and maximum come from those 2,000 chunks (the corpus's statistics from all)."""
    from oracle import weighted
    dev = device()
    n, n_docs, nq = 2000, 3000, 40
    ind, toks, csr, qi, qt = _small_corpus(6001, n_docs, 300, 30.0, nq)
    w = synth.mixture_dense(6002, n, 128, 16, nq, 10, "bf16")
    idx = make_index(w.rows, "bf16", capacity=n_docs)
    _attach(idx, csr, dev)
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    qt_oracle = np.where((qt >= 0) & (qt < 300), qt, 10 ** 6).astype(np.int64)
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    for k in (5, 100):
        log("weighted index smaller than its corpus", n, n_docs, k)
        sc, ids = idx.search_hybrid_weighted(w.queries.to(dev), _t(qi, dev), _t(qt, dev), 0.7, 0.3, k)
        torch.cuda.synchronize()
        _check_weighted(weighted.fused(S, B[:, :n], 0.7, 0.3), sc, ids, k, f"n={n} n_docs={n_docs} k={k}")


def test_weighted_fusion_past_the_lds_key_cache():
    """45,001 chunks, more than the 32,768 score keys the fusion kernel keeps in LDS: the
    steps past them compute the composites again from the score rows, and both halves must
    agree with the oracle (top-5 and top-100, every chunk in the sparse corpus)."""
    from oracle import weighted
    dev = device()
    n, nq = 45_001, 24
    ind, toks, csr, qi, qt = _small_corpus(4501, n, 500, 12.0, nq)
    w = synth.mixture_dense(4502, n, 128, 32, nq, 100, "bf16")
    idx = make_index(w.rows, "bf16")
    _attach(idx, csr, dev)
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    qt_oracle = np.where((qt >= 0) & (qt < 500), qt, 10 ** 6).astype(np.int64)
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)
    F = weighted.fused(S, B)
    for k in (5, 100):
        log("weighted past the LDS cache", n, k)
        sc, ids = idx.search_hybrid_weighted(w.queries.to(dev), _t(qi, dev), _t(qt, dev), 0.5, 0.5, k)
        torch.cuda.synchronize()
        _check_weighted(F, sc, ids, k, f"n={n} k={k}")


def test_weighted_fusion_index_growing_inside_a_larger_corpus():
    """A 40,000-chunk sparse corpus attached to an index of capacity 40,000 that holds 5,000,
    then 33,000, then 40,000 rows: the normalisation covers the chunks with a dense row only
    (the lexical minimum and maximum of the corpus's other chunks must not enter), and the
    workspace sized from the capacity serves every row count."""
    from paper_2608_08340_amd import OP_WEIGHTED
    from oracle import weighted
    dev = device()
    cap, nq = 40_000, 24
    ind, toks, csr, qi, qt = _small_corpus(5001, cap, 400, 14.0, nq)
    w = synth.mixture_dense(5002, cap, 128, 32, nq, 100, "bf16")
    idx = make_index(w.rows[:0], "bf16", capacity=cap)
    _attach(idx, csr, dev)
    ws = idx.workspace(OP_WEIGHTED, nq)
    qt_oracle = np.where((qt >= 0) & (qt < 400), qt, 10 ** 6).astype(np.int64)
    B = bm25.scores_batch(ind, toks, qi, qt_oracle, 1.2, 0.75)  # statistics over the whole corpus
    done = 0
    for n in (5_000, 33_000, 40_000):
        idx.upsert(w.rows[done:n].to(dev))
        done = n
        S, X, Q = oracle_scores(w.rows[:n], w.queries, "bf16")
        F = weighted.fused(S, B[:, :n])
        for k in (5, 100):
            log("weighted growing", n, k)
            sc, ids = idx.search_hybrid_weighted(w.queries.to(dev), _t(qi, dev), _t(qt, dev), 0.5, 0.5, k)
            torch.cuda.synchronize()
            assert idx.workspace(OP_WEIGHTED, nq).data_ptr() == ws.data_ptr()  # never regrown
            _check_weighted(F, sc, ids, k, f"n={n} k={k}")


@pytest.mark.timeout(300)
def test_weighted_fusion_32k(c3):
    """The 32,768 x 1,024 bf16 hybrid workload with weights 0.5 / 0.5, top-5, every query
    against the fp64 oracle."""
    from oracle import weighted
    dev = device()
    h = c3
    w = h.dense
    idx = make_index(w.rows, "bf16")
    _attach(idx, h.csr, dev, h.k1, h.b)
    sc, ids = idx.search_hybrid_weighted(w.queries.to(dev), _t(h.qterm_indptr, dev), _t(h.qterms, dev), 0.5, 0.5, 5)
    torch.cuda.synchronize()
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    B = bm25.scores_batch(h.doc_indptr, h.tokens, h.qterm_indptr, h.qterms, h.k1, h.b)
    _check_weighted(weighted.fused(S, B), sc, ids, 5, "32k weighted")
