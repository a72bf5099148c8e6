"""Seeded synthetic inputs shaped like the retrieval workload of the OpRAG paper.

The paper evaluates retrieval over 32K chunks derived from WikiText-103 with 1,024 query
sets (Section 5.1, setup); neither is available here, so every input is drawn from the
seeded generators below, with the shapes and value distributions stated per workload.

This module holds none of the retrieval arithmetic.  It draws random numbers, rounds them
to the storage dtype, and lays them out in the two formats the consumers need: raw token
sequences (what the oracle scans) and a CSR term -> (chunk, tf) matrix (what the library
takes).  Scoring, BM25 statistics, fusion and selection live in the library and,
independently, in the oracle.  Both sides receive the same stored bytes.

Seeds: ``numpy.random.SeedSequence([260808340, workload, stream, *sub])``.  Streams:
0 = mixture centres, 1 = rows, 2 = queries, 3 = sparse corpus, 4 = query terms,
10 + r = appended rows of streaming round r.
"""
from __future__ import annotations

import concurrent.futures as _cf
import os
from dataclasses import dataclass, field

import numpy as np
import torch

SEED_ROOT = 260808340

DTYPES = ("f32", "bf16", "f16")
_TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
_ELEM = {"f32": 4, "bf16": 2, "f16": 2}


def rng(workload: int, stream: int, *sub: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([SEED_ROOT, workload, stream, *sub]))


def elem_bytes(dtype: str) -> int:
    return _ELEM[dtype]


# --------------------------------------------------------------------------------------
# Dense vectors
# --------------------------------------------------------------------------------------

def _normalise(x: np.ndarray) -> np.ndarray:
    x /= np.linalg.norm(x, axis=1, keepdims=True).astype(np.float32)
    return x


def iid_unit_rows(g: np.random.Generator, n: int, d: int) -> np.ndarray:
    """n x d fp32 rows drawn i.i.d. N(0, 1) per coordinate, then L2-normalised."""
    return _normalise(g.standard_normal((n, d), dtype=np.float32))


def mixture_centres(g: np.random.Generator, n_clusters: int, d: int) -> np.ndarray:
    return g.standard_normal((n_clusters, d), dtype=np.float32)


def mixture_rows(g: np.random.Generator, centres: np.ndarray, n: int, sigma: float) -> np.ndarray:
    """Rows of a uniform-weight Gaussian mixture: normalise(centre + sigma * N(0, I)), fp32."""
    comp = g.integers(0, centres.shape[0], size=n)
    x = g.standard_normal((n, centres.shape[1]), dtype=np.float32)
    x *= np.float32(sigma)
    x += centres[comp]
    return _normalise(x)


def mixture_rows_chunked(workload: int, stream: int, centres: np.ndarray, n: int, sigma: float,
                         first_chunk: int = 0, chunk: int = 65536, threads: int | None = None) -> np.ndarray:
    """Large mixture draws, generated in independently seeded chunks of ``chunk`` rows.

    Chunk c of a stream uses seed (workload, stream, first_chunk + c), so the result does not
    depend on the thread count.
    """
    n_chunks = (n + chunk - 1) // chunk
    out = np.empty((n, centres.shape[1]), dtype=np.float32)

    def one(c: int) -> None:
        lo, hi = c * chunk, min(n, (c + 1) * chunk)
        out[lo:hi] = mixture_rows(rng(workload, stream, first_chunk + c), centres, hi - lo, sigma)

    threads = threads or min(16, os.cpu_count() or 1)
    with _cf.ThreadPoolExecutor(threads) as ex:
        list(ex.map(one, range(n_chunks)))
    return out


def perturbed_queries(g: np.random.Generator, rows: np.ndarray, nq: int, noise: float):
    """Queries that are noisy copies of randomly chosen rows.

    ``rows`` are the stored rows (upcast to fp32).  Each query is normalise(row + noise * N(0, I)).
    Returns (queries fp32 [nq x d], source row ids int64 [nq]).
    """
    src = g.integers(0, rows.shape[0], size=nq)
    q = rows[src].astype(np.float32, copy=True)
    q += np.float32(noise) * g.standard_normal(q.shape, dtype=np.float32)
    return _normalise(q), src.astype(np.int64)


def to_storage(x: np.ndarray, dtype: str) -> torch.Tensor:
    """Round fp32 values to the storage dtype (round-to-nearest-even), as a CPU tensor."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(_TORCH_DT[dtype]).contiguous()


def storage_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bits of a stored tensor: uint32 for fp32, uint16 for bf16 / fp16."""
    if t.dtype == torch.float32:
        return t.view(torch.int32).numpy().view(np.uint32)
    return t.view(torch.int16).numpy().view(np.uint16)


def upcast_f32(t: torch.Tensor) -> np.ndarray:
    """Stored tensor -> fp32 numpy (exact for bf16 / fp16)."""
    return t.to(torch.float32).numpy()


# --------------------------------------------------------------------------------------
# Sparse corpus
# --------------------------------------------------------------------------------------

def zipf_pmf(vocab: int, s: float) -> np.ndarray:
    """Finite Zipf law over term ids 0..vocab-1: P(term = r - 1) proportional to r^-s."""
    w = np.arange(1, vocab + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


def sparse_corpus(g: np.random.Generator, n_docs: int, vocab: int, s: float, mean_len: float):
    """Raw token sequences: Poisson(mean_len) lengths (at least 1), Zipf(s) tokens.

    Returns (doc_indptr int64 [n_docs + 1], tokens int32 [total]).
    """
    lens = np.maximum(g.poisson(mean_len, size=n_docs), 1).astype(np.int64)
    indptr = np.zeros(n_docs + 1, dtype=np.int64)
    np.cumsum(lens, out=indptr[1:])
    cdf = np.cumsum(zipf_pmf(vocab, s))
    u = g.random(int(indptr[-1]))
    tokens = np.minimum(np.searchsorted(cdf, u, side="right"), vocab - 1).astype(np.int32)
    return indptr, tokens


@dataclass
class CSR:
    """Term -> (chunk, tf) postings; chunk ids ascending within a term; tf >= 1."""
    term_indptr: np.ndarray  # int64 [vocab + 1]
    post_chunk: np.ndarray   # int32 [nnz]
    post_tf: np.ndarray      # int32 [nnz]
    doc_len: np.ndarray      # int32 [n_docs], tokens per chunk
    vocab: int
    n_docs: int

    @property
    def nnz(self) -> int:
        return int(self.post_chunk.shape[0])


def csr_from_tokens(doc_indptr: np.ndarray, tokens: np.ndarray, vocab: int) -> CSR:
    """Lay a raw token corpus out as the CSR postings matrix the library consumes."""
    n_docs = doc_indptr.shape[0] - 1
    lens = np.diff(doc_indptr)
    doc_of_tok = np.repeat(np.arange(n_docs, dtype=np.int64), lens)
    key = tokens.astype(np.int64) * n_docs + doc_of_tok
    uniq, counts = np.unique(key, return_counts=True)
    term = uniq // n_docs
    chunk = uniq % n_docs
    indptr = np.zeros(vocab + 1, dtype=np.int64)
    np.cumsum(np.bincount(term, minlength=vocab), out=indptr[1:])
    return CSR(indptr, chunk.astype(np.int32), counts.astype(np.int32), lens.astype(np.int32), vocab, n_docs)


def zipf_query_terms(g: np.random.Generator, nq: int, n_terms: int, vocab: int, s: float):
    """Each query gets n_terms i.i.d. Zipf(s) term ids (repeats allowed).

    Returns (qterm_indptr int32 [nq + 1], qterms int32 [nq * n_terms]).
    """
    cdf = np.cumsum(zipf_pmf(vocab, s))
    t = np.minimum(np.searchsorted(cdf, g.random(nq * n_terms), side="right"), vocab - 1)
    indptr = (np.arange(nq + 1, dtype=np.int64) * n_terms).astype(np.int32)
    return indptr, t.astype(np.int32)


def doc_query_terms(g: np.random.Generator, src: np.ndarray, doc_indptr: np.ndarray, tokens: np.ndarray,
                    n_terms: int):
    """Query terms drawn uniformly from the tokens of each query's source chunk (correlated variant)."""
    nq = src.shape[0]
    lo = doc_indptr[src]
    ln = doc_indptr[src + 1] - lo
    pos = lo[:, None] + (g.random((nq, n_terms)) * ln[:, None]).astype(np.int64)
    indptr = (np.arange(nq + 1, dtype=np.int64) * n_terms).astype(np.int32)
    return indptr, tokens[pos.reshape(-1)].astype(np.int32)


# --------------------------------------------------------------------------------------
# Workloads
# --------------------------------------------------------------------------------------

@dataclass
class DenseWorkload:
    name: str
    dtype: str
    rows: torch.Tensor           # stored rows [n x d], CPU
    queries: torch.Tensor        # stored queries [nq x d], CPU
    k: int
    src: np.ndarray | None = None
    extra: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return int(self.rows.shape[0])

    @property
    def d(self) -> int:
        return int(self.rows.shape[1])


def tiny_dense(n: int = 1024, d: int = 384, nq: int = 16, k: int = 5) -> DenseWorkload:
    """1,024 x 384 fp32 unit rows drawn i.i.d. N(0,1); 16 perturbed-copy queries (noise 0.1); top-5."""
    w = 1
    rows = to_storage(iid_unit_rows(rng(w, 1), n, d), "f32")
    q, src = perturbed_queries(rng(w, 2), upcast_f32(rows), nq, 0.1)
    return DenseWorkload("tiny_dense_1k_x_384_f32", "f32", rows, to_storage(q, "f32"), k, src)


def mixture_dense(workload: int, n: int, d: int, n_clusters: int, nq: int, k: int, dtype: str,
                  sigma: float = 0.3, name: str | None = None) -> DenseWorkload:
    """Unit rows from a uniform Gaussian mixture (centres N(0,1), within-cluster sigma), stored in
    ``dtype``; queries are perturbed copies (noise 0.1) of random stored rows."""
    centres = mixture_centres(rng(workload, 0), n_clusters, d)
    if n > 262144:
        rows32 = mixture_rows_chunked(workload, 1, centres, n, sigma)
    else:
        rows32 = mixture_rows(rng(workload, 1), centres, n, sigma)
    rows = to_storage(rows32, dtype)
    del rows32
    q, src = perturbed_queries(rng(workload, 2), upcast_f32(rows), nq, 0.1)
    nm = name or f"mixture_{n}_x_{d}_{dtype}"
    return DenseWorkload(nm, dtype, rows, to_storage(q, dtype), k, src, {"centres": centres, "sigma": sigma})


def dense_32k(nq: int = 1024, k: int = 5, n: int = 32768) -> DenseWorkload:
    """32,768 x 1,024 bf16 unit rows from a 256-component mixture (sigma 0.3); queries as above."""
    return mixture_dense(2, n, 1024, 256, nq, k, "bf16", name=f"dense_{n}_x_1024_bf16")


@dataclass
class HybridWorkload:
    dense: DenseWorkload
    doc_indptr: np.ndarray
    tokens: np.ndarray
    csr: CSR
    qterm_indptr: np.ndarray
    qterms: np.ndarray
    k_dense: int = 100
    k_sparse: int = 100
    rrf_k: int = 60
    k: int = 5
    k1: float = 1.2
    b: float = 0.75


def hybrid_32k(nq: int = 256, n: int = 32768, vocab: int = 30000, correlated: bool = False,
               dense: DenseWorkload | None = None) -> HybridWorkload:
    """The 32K x 1,024 bf16 dense index (the same rows and query draw as ``dense_32k``; the first
    ``nq`` queries) plus a synthetic sparse corpus: Zipf(1.1) terms over a 30,000-term vocabulary,
    Poisson(256) chunk lengths, 8 Zipf-drawn terms per query (or, with ``correlated``, 8 tokens of
    the query's source chunk)."""
    base = dense if dense is not None else dense_32k(n=n)
    dw = DenseWorkload(base.name.replace("dense", "hybrid"), base.dtype, base.rows,
                       base.queries[:nq].contiguous(), 100, base.src[:nq], base.extra)
    doc_indptr, tokens = sparse_corpus(rng(3, 3), dw.n, vocab, 1.1, 256.0)
    csr = csr_from_tokens(doc_indptr, tokens, vocab)
    if correlated:
        qi, qt = doc_query_terms(rng(3, 4), dw.src, doc_indptr, tokens, 8)
    else:
        qi, qt = zipf_query_terms(rng(3, 4), nq, 8, vocab, 1.1)
    return HybridWorkload(dw, doc_indptr, tokens, csr, qi, qt)
