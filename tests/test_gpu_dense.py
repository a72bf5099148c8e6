"""Dense exact top-k on the GPU against the fp64 oracle (parity), through the C ABI."""
import numpy as np
import pytest
import torch

import synth
from oracle import accept
from oracle import dense as od
from oracle.storage import decode
from tests.gpu_helpers import check_dense, device, log, make_index, oracle_scores

pytestmark = pytest.mark.gpu


def _run(rows, queries, k, dtype, capacity=None):
    dev = device()
    idx = make_index(rows, dtype, capacity)
    sc, ids = idx.search_dense(queries.to(dev), k)
    torch.cuda.synchronize()
    return idx, sc.cpu(), ids.cpu()


def test_read_probe_folds_every_word():
    """The read probe (diagnostics) reads every 16-byte word exactly once: the XOR of the
    workgroups' folds equals the XOR of the data (three workgroups, a ragged last stride)."""
    import paper_2608_08340_amd as P
    dev = device()
    g = torch.Generator().manual_seed(7)
    data = torch.randint(-2 ** 31, 2 ** 31 - 1, (1 << 16,), dtype=torch.int32, generator=g)
    sink = torch.zeros(3, dtype=torch.int32, device=dev)
    P.probe_read(data.to(dev), 3, sink)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(data.numpy().view(np.uint32))


def test_tiny_f32_1k_x_384():
    """1,024 x 384 fp32 rows, 16 perturbed queries, exact cosine top-5 (rtol 1e-5)."""
    device()
    w = synth.tiny_dense()
    log("tiny f32", tuple(w.rows.shape), w.k)
    _, sc, ids = _run(w.rows, w.queries, w.k, "f32")
    S, X, Q = oracle_scores(w.rows, w.queries, "f32")
    check_dense(S, X, Q, ids, sc, w.k, "f32")
    # the noisy copy of a chunk finds its source first at this size
    assert (ids[:, 0].numpy() == w.src).all()


@pytest.fixture(scope="module")
def c2():
    device()
    return synth.dense_32k()


@pytest.mark.parametrize("nq", [1, 16, 65, 128, 256, 384, 768, 1024])
def test_32k_x_1024_bf16_top5(c2, nq):
    """32,768 x 1,024 bf16 mixture rows; query batches 1, 16, 256, 384, 768, 1,024; exact
    top-5.  384 and 768 queries (three and six query blocks) get grids of fewer workgroups
    than CUs, with two and four tiles per chunk."""
    log("32k bf16 nq", nq)
    q = c2.queries[:nq].contiguous()
    _, sc, ids = _run(c2.rows, q, 5, "bf16")
    S, X, Q = oracle_scores(c2.rows, q, "bf16")
    reps = check_dense(S, X, Q, ids, sc, 5, "bf16")
    assert all(r.recall == 1.0 for r in reps)


@pytest.mark.parametrize("k", [8, 16])
def test_32k_x_1024_bf16_top8_top16_batch512(c2, k):
    """32,768 x 1,024 bf16, 512 queries, k = 8 and 16: the 128-query kernels with the running
    threshold on every tile after a chunk's first (two tiles per chunk at this batch)."""
    log("32k bf16 nq 512 k", k)
    q = c2.queries[:512].contiguous()
    _, sc, ids = _run(c2.rows, q, k, "bf16")
    S, X, Q = oracle_scores(c2.rows, q, "bf16")
    reps = check_dense(S, X, Q, ids, sc, k, "bf16")
    assert all(r.recall == 1.0 for r in reps)


@pytest.mark.parametrize("nq,k", [(1, 10), (1, 16), (16, 16), (64, 10), (64, 16), (100, 8), (100, 16), (128, 10)])
def test_32k_x_1024_bf16_small_batch_top10_top16(c2, nq, k):
    """32,768 x 1,024 bf16 at small batches with k = 10 and 16: 128 to 256 chunk lists of k
    entries per query, merged from one load batch of 64 composites per lane (sorted lists whose
    length divides 64, the case where lanes must not all see the same list position)."""
    log("32k bf16 nq", nq, "k", k)
    q = c2.queries[:nq].contiguous()
    _, sc, ids = _run(c2.rows, q, k, "bf16")
    S, X, Q = oracle_scores(c2.rows, q, "bf16")
    reps = check_dense(S, X, Q, ids, sc, k, "bf16")
    assert all(r.recall == 1.0 for r in reps)


@pytest.mark.parametrize("nq,k", [(1, 16), (16, 10), (50, 16)])
def test_long_list_merge_with_a_short_last_chunk(nq, k):
    """19,973 rows (156 full 128-row chunks and one of 5 rows, so one list holds fewer than k
    entries and is padded) at small batches: with k = 16, 2,512 composites per query, the
    workgroup-per-query merge; with k = 10, the one-wave merge of 1,570."""
    log("long list merge", nq, k)
    device()
    w = synth.mixture_dense(7300 + k + nq, 19973, 256, 48, nq, k, "bf16")
    _, sc, ids = _run(w.rows, w.queries, k, "bf16")
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    check_dense(S, X, Q, ids, sc, k, "bf16", label=f"nq={nq} k={k}")


@pytest.mark.parametrize("nq", [100, 256])
def test_32k_x_1024_bf16_top100(c2, nq):
    """The hybrid's dense list shape: 32,768 x 1,024 bf16, top-100 (filtered levels 2,048 ->
    32,768), at 100 queries (two 64-query blocks over 128-row tiles) and 256 (two 128-query
    blocks)."""
    log("32k bf16 top-100 nq", nq)
    q = c2.queries[:nq].contiguous()
    _, sc, ids = _run(c2.rows, q, 100, "bf16")
    S, X, Q = oracle_scores(c2.rows, q, "bf16")
    reps = check_dense(S, X, Q, ids, sc, 100, "bf16")
    assert all(r.recall == 1.0 for r in reps)


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
@pytest.mark.parametrize("k", [1, 5, 16, 100])
def test_exact_integer_scores_and_ties(dtype, k):
    """Small-integer vectors give exact dot products with many exact ties: ids must match the
    oracle exactly, ties by ascending id."""
    device()
    g = np.random.default_rng(1000 + k)
    n, d, nq = 3001, 128, 37
    X = g.integers(-2, 3, size=(n, d)).astype(np.float32)
    Q = g.integers(-2, 3, size=(nq, d)).astype(np.float32)
    rows, qs = synth.to_storage(X, dtype), synth.to_storage(Q, dtype)
    _, sc, ids = _run(rows, qs, k, dtype)
    S = Q.astype(np.float64) @ X.astype(np.float64).T
    ref_ids, ref_sc = od.topk_from_scores(S, k)
    assert np.array_equal(ids.numpy(), ref_ids)
    assert np.array_equal(sc.numpy().astype(np.float64), ref_sc)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("n,nq,k", [(3000, 1, 7), (3000, 17, 8), (3000, 65, 9), (2500, 130, 16), (3000, 40, 17),
                                    (4100, 33, 64), (5000, 70, 100), (3000, 9, 128), (64, 5, 100), (1, 3, 4),
                                    (9000, 21, 40), (20000, 130, 128)])
def test_ragged_sizes_and_k(dtype, n, nq, k):
    """Row counts that are not tile multiples, query counts that are not block multiples, k across
    both selection strategies, k larger than the index (padding)."""
    device()
    w = synth.mixture_dense(200 + n % 97, n, 128, 16, nq, k, dtype)
    _, sc, ids = _run(w.rows, w.queries, k, dtype)
    S, X, Q = oracle_scores(w.rows, w.queries, dtype)
    check_dense(S, X, Q, ids, sc, k, dtype, label=f"n={n} nq={nq} k={k}")


def _sweep_cases(n_cases=40, seed=2608):
    """Seeded (dtype, n, d, nq, k) draws across the kernel table: dimensions whose k-step count
    admits rings of 4, 8 or 16 (or only 4), query blocks resident or streamed, the largest
    dimension, every batch class and both selection strategies."""
    r = np.random.default_rng(seed)
    dims = [128, 256, 384, 640, 896, 1024, 1152, 2048, 4096, 8192]
    batches = [1, 2, 5, 16, 17, 40, 64, 65, 100, 128, 129, 200, 256, 300, 513]
    ks = [1, 2, 5, 6, 8, 9, 16, 17, 33, 100, 128]
    out = []
    for i in range(n_cases):
        d = dims[i % len(dims)]
        nq = int(r.choice(batches))
        k = int(r.choice(ks))
        n = int(r.integers(300, 5000)) if d <= 2048 else int(r.integers(200, 1500))
        out.append(("bf16" if i % 3 else "f16", n, d, nq, k))
    return out


@pytest.mark.parametrize("dtype,n,d,nq,k", _sweep_cases())
def test_seeded_shape_sweep(dtype, n, d, nq, k):
    """Parity over seeded shapes that reach every ring depth, resident and streamed query
    blocks, d up to the largest supported dimension, ragged rows and batches, k on both sides
    of the list/threshold boundary."""
    log("sweep", dtype, n, d, nq, k)
    device()
    w = synth.mixture_dense(500 + d // 128 + nq, n, d, 24, nq, k, dtype)
    _, sc, ids = _run(w.rows, w.queries, k, dtype)
    S, X, Q = oracle_scores(w.rows, w.queries, dtype)
    check_dense(S, X, Q, ids, sc, k, dtype, label=f"{dtype} n={n} d={d} nq={nq} k={k}")


@pytest.mark.parametrize("d", [512, 1536])
@pytest.mark.parametrize("nq", [1, 16])
def test_small_batch_resident_and_streamed_queries(d, nq):
    """The batch-1 to 16 top-5 kernel keeps its query block resident in LDS up to 1,024
    dimensions: d = 512 fills four of its eight slices; d = 1,536 takes the streamed kernel."""
    device()
    w = synth.mixture_dense(300 + d // 128, 5000, d, 16, nq, 5, "bf16")
    _, sc, ids = _run(w.rows, w.queries, 5, "bf16")
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    check_dense(S, X, Q, ids, sc, 5, "bf16", label=f"d={d} nq={nq}")


@pytest.mark.parametrize("kind", ["ints", "four_rows"])
@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("nq,k", [(1, 7), (16, 5), (40, 16), (130, 5), (130, 10)])
def test_multi_tile_chunks_exact_ties(kind, dtype, nq, k):
    """393,293 x 128 integer rows: enough rows that every query block walks several tiles per
    row chunk, so the selection runs against running thresholds.  "ints": entries in
    {-2..2}, exact scores with ties near the k-th value.  "four_rows": every row is one of four
    vectors, so each tile holds dozens of rows tied at the best score and the tie handling
    takes its overflow paths.  Ids and scores must equal the oracle's exactly."""
    device()
    g = np.random.default_rng(7000 + 31 * nq + k + (0 if kind == "ints" else 1))
    n, d = 393_216 + 77, 128
    if kind == "ints":
        X = g.integers(-2, 3, size=(n, d)).astype(np.float32)
    else:
        X = g.integers(-2, 3, size=(4, d)).astype(np.float32)[g.integers(0, 4, size=n)]
    Q = g.integers(-2, 3, size=(nq, d)).astype(np.float32)
    log("multi-tile", kind, dtype, nq, k)
    _, sc, ids = _run(synth.to_storage(X, dtype), synth.to_storage(Q, dtype), k, dtype)
    samp = np.unique(np.r_[0:min(nq, 12), nq - 1])
    S = Q[samp].astype(np.float64) @ X.astype(np.float64).T
    ref_ids, ref_sc = od.topk_from_scores(S, k)
    assert np.array_equal(ids.numpy()[samp], ref_ids)
    assert np.array_equal(sc.numpy()[samp].astype(np.float64), ref_sc)


@pytest.mark.parametrize("nq,k", [(1, 16), (16, 16), (3, 5), (40, 8)])
def test_merge_with_candidates_concentrated(nq, k):
    """32,768 rows where every fourth run of 64 rows scores high and the rest low: the best
    entries of many per-chunk lists compete, so the list merge sees far more composites above
    its threshold than one wave can rank at once and extracts the k best one at a time.
    Integer values: ids and scores must equal the oracle's exactly."""
    device()
    n, d = 32_768, 128
    r = np.arange(n)
    X = np.zeros((n, d), np.float32)
    X[:, 0] = np.where((r // 64) % 4 == 0, 100 + r % 37, r % 50)
    X[:, 1:] = np.random.default_rng(5).integers(-1, 2, size=(n, d - 1))
    Q = np.zeros((nq, d), np.float32)
    Q[:, 0] = 1.0
    Q[:, 1] = np.arange(nq) % 3 - 1  # small query-dependent perturbation
    log("concentrated", nq, k)
    _, sc, ids = _run(synth.to_storage(X, "bf16"), synth.to_storage(Q, "bf16"), k, "bf16")
    S = Q.astype(np.float64) @ X.astype(np.float64).T
    ref_ids, ref_sc = od.topk_from_scores(S, k)
    assert np.array_equal(ids.numpy(), ref_ids)
    assert np.array_equal(sc.numpy().astype(np.float64), ref_sc)


@pytest.mark.parametrize("nq", [3, 70])
@pytest.mark.parametrize("case", ["repair", "fallback"])
def test_filtered_overflow_repair(case, nq):
    """k > 16 runs in threshold levels with candidate buffers of max(4,096, 256 k) keys.
    "repair": the first 4,096 rows score low, so the last level's threshold admits ~56,000
    rows and the buffers overflow; the device-side repair reruns the last level with the
    k-th scores found so far.  "fallback": a quarter of 120,000 rows tie at the top score,
    so every repair overflows too and the per-chunk-list plan answers.  Exact either way."""
    device()
    g = np.random.default_rng(11 + nq)
    k, d = 17, 128
    if case == "repair":
        n = 60_000
        r = np.arange(n)
        X = np.zeros((n, d), np.float32)
        X[:, 0] = np.where(r < 4096, r % 7, 20 + (r * 7919) % 200)  # integers < 256: exact in bf16
    else:
        n = 120_000
        X = g.integers(-2, 3, size=(4, d)).astype(np.float32)[g.integers(0, 4, size=n)]
    X[:, 1] = g.integers(-1, 2, size=n)
    Q = np.zeros((nq, d), np.float32)
    Q[:, 0] = 1.0
    Q[:, 2:] = g.integers(0, 2, size=(nq, d - 2)) if case == "fallback" else 0.0
    log("overflow", case, nq)
    _, sc, ids = _run(synth.to_storage(X, "bf16"), synth.to_storage(Q, "bf16"), k, "bf16")
    S = Q.astype(np.float64) @ X.astype(np.float64).T
    ref_ids, ref_sc = od.topk_from_scores(S, k)
    assert np.array_equal(ids.numpy(), ref_ids)
    assert np.array_equal(sc.numpy().astype(np.float64), ref_sc)


@pytest.mark.parametrize("k", [17, 100])
def test_workspace_sized_from_capacity_covers_every_row_count(k):
    """The workspace size a search reports depends on the capacity only.  Filtered searches
    keep every row in their buffers up to 32,768 rows (no repair launches) and switch to
    max(4,096, 256 k) slots per query above, so a workspace sized for a 60,000-row capacity
    must still cover 32,768 rows: the index grows through both regimes with one workspace."""
    dev = device()
    from paper_2608_08340_amd import OP_DENSE
    cap, d, nq = 60_000, 128, 40
    w = synth.mixture_dense(900 + k, cap, d, 32, nq, k, "bf16")
    idx = make_index(w.rows[:0], "bf16", capacity=cap)
    need = idx.workspace_bytes(OP_DENSE, nq, k)
    ws = idx.workspace(OP_DENSE, nq, k)
    assert ws.numel() == need
    done = 0
    for n in (5_000, 32_768, 40_000, 60_000):
        idx.upsert(w.rows[done:n].to(dev))
        done = n
        log("capacity workspace", k, n)
        sc, ids = idx.search_dense(w.queries.to(dev), k)
        assert idx.workspace(OP_DENSE, nq, k).data_ptr() == ws.data_ptr()  # never regrown
        S, X, Q = oracle_scores(w.rows[:n], w.queries, "bf16")
        check_dense(S, X, Q, ids, sc, k, "bf16", label=f"n={n} k={k}")


def test_empty_index_pads():
    dev = device()
    from paper_2608_08340_amd import Index
    idx = Index(128, 100, torch.bfloat16)
    q = synth.to_storage(np.ones((3, 128), np.float32), "bf16").to(dev)
    sc, ids = idx.search_dense(q, 5)
    torch.cuda.synchronize()
    assert (ids.cpu() == -1).all() and torch.isneginf(sc.cpu()).all()


def test_repeatable_batch_invariant_prefix_consistent(c2):
    dev = device()
    idx = make_index(c2.rows, "bf16")
    q = c2.queries[:300].to(dev)
    s1, i1 = idx.search_dense(q, 10)
    s2, i2 = idx.search_dense(q, 10)
    s3, i3 = idx.search_dense(q[100:140].contiguous(), 10)
    s5, i5 = idx.search_dense(q, 5)
    torch.cuda.synchronize()
    assert torch.equal(i1, i2) and torch.equal(s1.view(torch.int32), s2.view(torch.int32))
    assert torch.equal(i3, i1[100:140]) and torch.equal(s3, s1[100:140])
    assert torch.equal(i5, i1[:, :5]) and torch.equal(s5, s1[:, :5])


def test_large_query_batch():
    """A large query batch (33,000 queries over 512 rows)."""
    device()
    w = synth.mixture_dense(300, 512, 128, 8, 33000, 3, "bf16")
    _, sc, ids = _run(w.rows, w.queries, 3, "bf16")
    S, X, Q = oracle_scores(w.rows, w.queries, "bf16")
    sel = np.r_[0:50, 32700:33000]
    check_dense(S[sel], X, Q[sel], ids[sel], sc[sel], 3, "bf16", strict=False)


def certify_all(Xb, dtype, Q, ids, sc, k, n, samp=None, step=1 << 16):
    """Sort-free certificate for every query against fp64 scores of every stored row.

    One pass over the rows in blocks (fp64 GEMM on the host's BLAS threads): the rows that
    are not returned and score above a query's k-th returned score plus its bound are
    collected, with their own bounds, and none may beat the k-th by more than both bounds.
    Also returns the fp64 score rows of the queries in ``samp`` (for the full-sort check)."""
    nq, d = Q.shape
    valid = ids >= 0
    Xr = decode(Xb[np.where(valid, ids, 0).reshape(-1)], dtype).reshape(nq, k, d)
    s_ret = np.where(valid, np.einsum("qkd,qd->qk", Xr, Q), 0.0)
    err = accept.strict_err(np.einsum("qkd,qd->qk", np.abs(Xr), np.abs(Q)), d)
    kk = min(k, n)
    j = np.argmin(np.where(np.arange(k) < kk, s_ret, np.inf), axis=1)
    thr = s_ret[np.arange(nq), j] + err[np.arange(nq), j]
    S_samp = None if samp is None else np.empty((len(samp), n))
    hits_q, hits_r, hits_s = [], [], []
    for lo in range(0, n, step):
        hi = min(n, lo + step)
        Sc = od.scores(decode(Xb[lo:hi], dtype), Q)
        if samp is not None:
            S_samp[:, lo:hi] = Sc[samp]
        rows = ids - lo
        m = valid & (rows >= 0) & (rows < hi - lo)
        qq = np.nonzero(m)[0]
        Sc[qq, rows[m]] = -np.inf  # returned rows
        hq, hr = np.nonzero(Sc > thr[:, None])
        hits_q.append(hq)
        hits_r.append(hr + lo)
        hits_s.append(Sc[hq, hr])
    hq, hr, hs = np.concatenate(hits_q), np.concatenate(hits_r), np.concatenate(hits_s)
    he = accept.strict_err(np.einsum("nd,nd->n", np.abs(decode(Xb[hr], dtype)), np.abs(Q[hq])), d)
    for q in range(nq):
        m = hq == q
        rep = accept.certificate(s_ret[q], ids[q], sc[q], err[q], k, n, s_unreturned=hs[m], err_unreturned=he[m])
        assert rep.ok, (q, rep.problems)
    return S_samp, len(hq)


@pytest.mark.timeout(600)
def test_1m_x_768_bf16_top10_sampled():
    """1,048,576 x 768 bf16 rows (4,096-cluster mixture), 1,024 queries, exact top-10.
    Every query: fp64 scores of every row, the returned scores within the fp32 bound, list
    order, and no unreturned row above the k-th returned score beyond both bounds; 64 sampled
    queries: the full acceptance rules against a sort of every row within 0.05 of the oracle's
    own 10th best score (found by a partition of all rows)."""
    dev = device()
    log("generating 1M x 768")
    n = 1 << 20
    w = synth.mixture_dense(4, n, 768, 4096, 1024, 10, "bf16")
    idx = make_index(w.rows, "bf16")
    sc, ids = idx.search_dense(w.queries.to(dev), 10)
    torch.cuda.synchronize()
    sc, ids = sc.cpu().numpy(), ids.cpu().numpy()
    log("certifying every query")
    Xb = synth.storage_bits(w.rows)
    Q = decode(synth.storage_bits(w.queries), "bf16")
    samp = np.random.default_rng(4).choice(1024, 64, replace=False)
    S, n_close = certify_all(Xb, "bf16", Q, ids, sc, 10, n, samp=samp)
    log(f"unreturned rows within the bounds of a k-th score: {n_close}")
    # rows within 0.05 of the oracle's own 10th best take part in the full check (every other
    # row is far below the top 10: it may be neither returned nor missed)
    kth = -np.partition(-S, 9, axis=1)[:, 9]
    reps = accept.check_batch(S, ids[samp], sc[samp], 10, rtol=2e-3, ranked=S >= (kth - 0.05)[:, None])
    assert all(r.ok for r in reps), [r.problems for r in reps if not r.ok][:2]
