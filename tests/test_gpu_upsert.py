"""Append-only upsert on the GPU: stored bytes, capacity handling, visibility to later searches
on the same stream, and streaming rounds of upsert + exact top-100 search."""
import os

import numpy as np
import pytest
import torch

import synth
from oracle import accept
from oracle import dense as od
from oracle.storage import decode, round_f32_to_bf16, round_f32_to_f16
from oracle.upsert import HostIndex
from tests.gpu_helpers import DT, check_dense, device, log

pytestmark = pytest.mark.gpu


def _hard_f32(g, m, d):
    x = (g.standard_normal((m, d)) * 10.0 ** g.integers(-8, 8, (m, d))).astype(np.float32)
    # exact round-to-nearest-even ties for bf16 and fp16
    u = x.view(np.uint32)
    u[0, : d // 2] = (u[0, : d // 2] & 0xFFFF0000) | 0x8000
    u[1, : d // 2] = (u[1, : d // 2] & 0xFFFFE000) | 0x1000
    x[2, :4] = [0.0, -0.0, 65504.0, 1e-8]
    return x


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_fp32_rows_are_rounded_to_nearest_even(dtype):
    dev = device()
    from paper_2608_08340_amd import Index
    g = np.random.default_rng(5)
    x = _hard_f32(g, 300, 128)
    idx = Index(128, 1000, DT[dtype])
    host = HostIndex(128, 1000, dtype)
    assert idx.upsert(torch.from_numpy(x).to(dev)) == 0 == host.append_f32(x)
    assert idx.upsert(torch.from_numpy(x[:7]).to(dev)) == 300 == host.append_f32(x[:7])
    torch.cuda.synchronize()
    got = idx.slab[:307].cpu().view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, host.valid_bits())
    assert idx.n_rows == 307


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_same_dtype_copy_is_bit_exact(dtype):
    dev = device()
    from paper_2608_08340_amd import Index
    x = synth.to_storage(np.random.default_rng(6).standard_normal((257, 128)).astype(np.float32), dtype)
    idx = Index(128, 600, DT[dtype])
    idx.upsert(x.to(dev))
    idx.upsert(x[:100].contiguous().to(dev))
    torch.cuda.synchronize()
    assert torch.equal(idx.slab[:257].cpu(), x) and torch.equal(idx.slab[257:357].cpu(), x[:100])


def test_capacity_is_all_or_nothing():
    dev = device()
    from paper_2608_08340_amd import Index, OpragError
    idx = Index(128, 100, torch.bfloat16)
    a = torch.randn(90, 128, device=dev).to(torch.bfloat16)
    idx.upsert(a)
    torch.cuda.synchronize()
    before = idx.slab.clone()
    with pytest.raises(OpragError) as e:
        idx.upsert(torch.randn(11, 128, device=dev).to(torch.bfloat16))
    assert e.value.status == -2
    torch.cuda.synchronize()
    assert idx.n_rows == 90 and torch.equal(idx.slab, before)
    assert idx.upsert(torch.randn(10, 128, device=dev).to(torch.bfloat16)) == 90
    with pytest.raises(OpragError):
        idx.upsert(torch.randn(1, 128, device=dev))      # fp32 into a full index
    with pytest.raises(OpragError):
        idx.upsert(torch.randn(2, 32, device=dev).to(torch.bfloat16))  # wrong width


def test_new_rows_visible_to_search_on_the_same_stream():
    dev = device()
    from paper_2608_08340_amd import Index
    w = synth.mixture_dense(71, 6000, 256, 32, 8, 5, "bf16")
    idx = Index(256, 7000, torch.bfloat16)
    idx.upsert(w.rows[:5000].to(dev))
    new = w.rows[5000:].to(dev)
    first = idx.upsert(new)                      # enqueued, no sync before the search
    sc, ids = idx.search_dense(new[::50].contiguous(), 1)
    torch.cuda.synchronize()
    assert first == 5000
    assert (ids[:, 0].cpu().numpy() == np.arange(5000, 6000, 50)).all()


def _full_scores(bits, n, Q, step=1 << 18):
    """fp64 oracle scores of every stored fp16 row [0, n) against Q, one block per task."""
    import concurrent.futures as cf
    S = np.empty((Q.shape[0], n))

    def block(lo):
        S[:, lo:min(n, lo + step)] = od.scores(decode(bits[lo:min(n, lo + step)], "f16"), Q)

    with cf.ThreadPoolExecutor(min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(block, range(0, n, step)))
    return S


def _streaming(n0, rounds, m, d, clusters, nq, k, sample, workload=5):
    """Start from n0 fp16 rows, then per round append m rows (the same generator) and search
    nq fresh queries drawn from the current rows, exact top-k."""
    dev = device()
    from paper_2608_08340_amd import Index
    cen = synth.mixture_centres(synth.rng(workload, 0), clusters, d)
    cap = n0 + rounds * m
    log("streaming: generating", n0, "rows")
    host = synth.mixture_rows_chunked(workload, 1, cen, n0, 0.3)
    rows_cpu = synth.to_storage(host, "f16")
    del host
    bits = np.empty((cap, d), dtype=np.uint16)
    bits[:n0] = synth.storage_bits(rows_cpu)
    idx = Index(d, cap, torch.float16)
    idx.upsert(rows_cpu.to(dev))
    del rows_cpu
    n = n0
    for r in range(rounds):
        new32 = synth.mixture_rows_chunked(workload, 10 + r, cen, m, 0.3)
        first = idx.upsert(torch.from_numpy(new32).to(dev))      # fp32 in, rounded on the GPU
        bits[n:n + m] = round_f32_to_f16(new32)                  # the oracle's own rounding
        assert first == n
        n += m
        cur = decode(bits[np.random.default_rng(r).integers(0, n, nq)], "f16").astype(np.float32)
        q32, _ = synth.perturbed_queries(synth.rng(workload, 2, r), cur, nq, 0.1)
        q = synth.to_storage(q32, "f16")
        sc, ids = idx.search_dense(q.to(dev), k)
        # self-queries of appended rows find themselves
        self_q = idx.slab[n - m:n - m + 64].clone()
        ssc, sids = idx.search_dense(self_q, 1)
        torch.cuda.synchronize()
        assert np.array_equal(idx.slab[n - m:n].cpu().view(torch.int16).numpy().view(np.uint16), bits[n - m:n])
        assert (sids[:, 0].cpu().numpy() == np.arange(n - m, n - m + 64)).all()
        sc, ids = sc.cpu().numpy(), ids.cpu().numpy()
        Q = decode(synth.storage_bits(q), "f16")
        # every query: fp64 score of each returned row, list length and order
        valid = ids >= 0
        Xr = decode(bits[np.where(valid, ids, 0).reshape(-1)], "f16").reshape(nq, k, d)
        s_ret = np.where(valid, np.einsum("qkd,qd->qk", Xr, Q), 0.0)
        err = accept.strict_err(np.einsum("qkd,qd->qk", np.abs(Xr), np.abs(Q)), d)
        for qq in range(nq):
            rep = accept.certificate(s_ret[qq], ids[qq], sc[qq], err[qq], k, n)
            assert rep.ok, (r, qq, rep.problems)
        # sampled queries: full oracle (row blocks scored on a thread pool).  Only rows within
        # 0.05 of the oracle's own k-th best score take part in the ranking (found by a
        # partition): every other row is far below the top k, so it may be neither returned
        # nor missed, and the full check sorts thousands of rows instead of all of them.
        samp = np.random.default_rng(100 + r).choice(nq, sample, replace=False)
        S = _full_scores(bits, n, Q[samp])
        kth = -np.partition(-S, k - 1, axis=1)[:, k - 1]
        reps = accept.check_batch(S, ids[samp], sc[samp], k, rtol=2e-3, ranked=S >= (kth - 0.05)[:, None])
        assert all(rp.ok for rp in reps), (r, [rp.problems for rp in reps if not rp.ok][:2])
        log(f"round {r}: n_rows {n} ok")


def test_streaming_upsert_and_search_small():
    _streaming(n0=131072, rounds=4, m=16384, d=384, clusters=512, nq=512, k=100, sample=16, workload=55)


@pytest.mark.timeout(1200)
def test_streaming_8m_x_384_f16_top100_full_size():
    """8,388,608 x 384 fp16 rows (8,192 clusters), 16 rounds of +65,536 rows and 4,096 queries, top-100.
    Every query of every round: returned scores against fp64, list length and order; 16
    sampled queries per round: fp64 scores of every row and the full acceptance rules over the
    rows within 0.05 of the oracle's own 100th best score."""
    _streaming(n0=8388608, rounds=16, m=65536, d=384, clusters=8192, nq=4096, k=100, sample=16)


def _ulp(x: np.ndarray, dtype: str) -> np.ndarray:
    """One unit in the last place of the storage dtype at |x| (normal range)."""
    mant = {"bf16": 7, "f16": 10, "f32": 23}[dtype]
    e = np.floor(np.log2(np.maximum(np.abs(x), 1e-30)))
    return np.exp2(e - mant)


@pytest.mark.parametrize("dtype,hidden_dtype,d", [(a, b, 128) for a in ("bf16", "f16", "f32") for b in ("bf16", "f32")]
                         + [("bf16", "bf16", 1152), ("f32", "f32", 260)])
def test_pooled_upsert_matches_mean_pool_l2_oracle(dtype, hidden_dtype, d):
    """Embedding tail fused with the upsert: 45 chunks of up to 50 hidden states of width d
    (128; 1,152 = one full and one partial block of 1,024 dimensions; 260, not a multiple of
    eight, for the element-wise path) (lengths include 0, 1, T, above T and negative, clamped to [0, T]), appended after 11
    existing rows.  Each stored element is within one unit in the last place of the storage
    dtype, plus the fp32 summation bound len * 2^-24 * sum|h| / ||sum||, of the fp64 mean-pool
    + L2 oracle; zero chunks are stored as zeros, and a pooled row used as a query finds
    itself."""
    from oracle import embed_tail
    from paper_2608_08340_amd import Index
    dev = device()
    g = np.random.default_rng(77)
    m, T = 45, 50
    H = g.standard_normal((m, T, d)).astype(np.float32) + 0.3
    lengths = g.integers(1, T + 1, size=m).astype(np.int32)
    lengths[:6] = [0, 1, T, T + 9, -3, 2]
    H[5, :2] = 0.0  # zero sum
    Ht = torch.from_numpy(H)
    if hidden_dtype == "bf16":
        Ht = Ht.to(torch.bfloat16)
    H64 = Ht.float().numpy().astype(np.float64)
    idx = Index(d, 100, DT[dtype])
    base = g.standard_normal((11, d))
    base /= np.linalg.norm(base, axis=1, keepdims=True)
    idx.upsert(synth.to_storage(base.astype(np.float32), dtype).to(dev))
    log("pooled upsert", dtype, hidden_dtype)
    first = idx.upsert_pooled(Ht.to(dev), torch.from_numpy(lengths).to(dev))
    torch.cuda.synchronize()
    assert first == 11 and idx.n_rows == 11 + m
    got = decode(synth.storage_bits(idx.slab[11:11 + m].cpu()), dtype)
    ref = embed_tail.pool(H64, lengths)
    n = np.clip(lengths, 0, T)
    bound = np.zeros_like(ref)
    for i in range(m):
        if n[i] == 0:
            continue
        tot = H64[i, : n[i]].sum(axis=0)
        nrm = np.linalg.norm(tot)
        if nrm > 0:
            bound[i] = 2 * n[i] * 2.0 ** -24 * np.abs(H64[i, : n[i]]).sum(axis=0) / nrm
    err = np.abs(got - ref)
    tol = _ulp(ref, dtype) * (ref != 0) + bound
    assert np.all(err <= tol), float(np.max(err - tol))
    assert np.all(got[[0, 4, 5]] == 0.0)
    norms = np.linalg.norm(got[6:], axis=1)
    assert np.allclose(norms, 1.0, atol=4 * {"bf16": 2 ** -8, "f16": 2 ** -11, "f32": 2 ** -23}[dtype])
    if dtype != "f32":
        q = idx.slab[11 + 10:11 + 14].clone()
        sc, ids = idx.search_dense(q, 1)
        torch.cuda.synchronize()
        assert ids[:, 0].cpu().tolist() == [21, 22, 23, 24]
