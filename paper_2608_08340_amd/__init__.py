"""MI355X-native exact-retrieval core of OpRAG: Python binding of liboprag.so.

The binding only marshals arguments: every step of upsert and search runs in the HIP
kernels behind the C ABI of ``include/oprag.h``.  PyTorch provides device memory and the
current stream.  Importing the package needs nothing built; the first call that reaches
the library raises ``OpragError`` if ``liboprag.so`` is missing (build it with
``paper_2608_08340_amd.build.build()``).

    idx = Index(dim=1024, capacity=32768, dtype=torch.bfloat16)
    idx.upsert(rows)                                   # Op_upsert
    scores, ids = idx.search_dense(queries, k=5)       # Op_retrieve, exact top-k
    idx.attach_sparse(term_indptr, post_chunk, post_tf, doc_len)
    fused, ids = idx.search_hybrid(queries, qterm_indptr, qterms)
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

__all__ = ["Index", "OpragError", "rrf_fuse", "library", "LIB_PATH", "OP_DENSE", "OP_SPARSE", "OP_HYBRID",
           "OP_DENSE_FIRST", "OP_WEIGHTED"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liboprag.so")
OP_DENSE, OP_SPARSE, OP_HYBRID, OP_DENSE_FIRST, OP_WEIGHTED = 0, 1, 2, 3, 4
_DTYPE = {torch.float32: 0, torch.bfloat16: 1, torch.float16: 2}
STATUS = {0: "OK", -1: "E_INVALID", -2: "E_CAPACITY", -3: "E_STATE", -4: "E_UNSUPPORTED", -5: "E_DEVICE"}


class OpragError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class _Desc(ctypes.Structure):
    _fields_ = [("dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("capacity", ctypes.c_int64),
                ("device", ctypes.c_int32), ("reserved", ctypes.c_int32)]


_P = ctypes.c_void_p
_I32, _I64, _SZ, _F = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
_SIGS = {
    "oprag_abi_version": ([], _I32),
    "oprag_last_error": ([], ctypes.c_char_p),
    "oprag_index_create": ([ctypes.POINTER(_Desc), _P, _SZ, ctypes.POINTER(_P)], _I32),
    "oprag_index_destroy": ([_P], _I32),
    "oprag_index_size": ([_P, ctypes.POINTER(_I64)], _I32),
    "oprag_upsert": ([_P, _P, _I32, _I64, _P, ctypes.POINTER(_I64)], _I32),
    "oprag_sparse_attach": ([_P, _I32, _I64, _I64, _P, _P, _P, _P, _F, _F, _P], _I32),
    "oprag_workspace_bytes": ([_P, _I32, _I64, _I32, _I32, ctypes.POINTER(_SZ)], _I32),
    "oprag_search_dense": ([_P, _P, _I64, _I32, _P, _P, _P, _SZ, _P], _I32),
    "oprag_search_dense_noalloc": ([_P, _P, _I64, _I32, _P, _P, _P], _I32),
    "oprag_search_sparse": ([_P, _P, _P, _I64, _I32, _P, _P, _P, _SZ, _P], _I32),
    "oprag_rrf_fuse": ([_P, _I32, _P, _I32, _I64, _I32, _I32, _P, _P, _P], _I32),
    "oprag_search_hybrid": ([_P, _P, _I64, _P, _P, _I32, _I32, _I32, _I32, _P, _P, _P, _SZ, _P], _I32),
    "oprag_search_hybrid_dense_first": ([_P, _P, _I64, _P, _P, _I32, _I32, _I32, _P, _P, _P, _SZ, _P], _I32),
    "oprag_upsert_pooled": ([_P, _P, _I32, _P, _I64, _I32, _P, ctypes.POINTER(_I64)], _I32),
    "oprag_search_hybrid_weighted": ([_P, _P, _I64, _P, _P, ctypes.c_float, ctypes.c_float, _I32, _P, _P, _P, _SZ, _P],
                                     _I32),
    "oprag_time_next_dense_kernel": ([_P, _P], _I32),
    "oprag_probe_read": ([_P, _SZ, _I32, _P, _P], _I32),
}
_lib = None
_lock = threading.Lock()


def library() -> ctypes.CDLL:
    """The loaded liboprag.so (raises OpragError when it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise OpragError(-4, f"{LIB_PATH} is not built; run paper_2608_08340_amd.build.build()")
            lib = ctypes.CDLL(LIB_PATH)
            for name, (args, res) in _SIGS.items():
                fn = getattr(lib, name)
                fn.argtypes = args
                fn.restype = res
            _lib = lib
    return _lib


def _check(status: int) -> None:
    if status != 0:
        raise OpragError(status, library().oprag_last_error().decode())


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dev_tensor(t: torch.Tensor, dtype, device, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or t.device != device or not t.is_contiguous():
        raise OpragError(-1, f"{name} must be a contiguous {dtype} tensor on {device}")
    return t


class Index:
    """An exact-retrieval index over a preallocated HBM slab of ``capacity`` rows."""

    def __init__(self, dim: int, capacity: int, dtype: torch.dtype = torch.bfloat16, device: int = 0):
        if dtype not in _DTYPE:
            raise OpragError(-1, f"unsupported dtype {dtype}")
        lib = library()
        self.dim, self.capacity, self.dtype = int(dim), int(capacity), dtype
        self.device = torch.device("cuda", device)
        self.slab = torch.empty((self.capacity, self.dim), dtype=dtype, device=self.device)
        desc = _Desc(self.dim, _DTYPE[dtype], self.capacity, device, 0)
        h = ctypes.c_void_p()
        _check(lib.oprag_index_create(ctypes.byref(desc), _ptr(self.slab),
                                      self.slab.numel() * self.slab.element_size(), ctypes.byref(h)))
        self._h = h
        self._ws = torch.empty(0, dtype=torch.uint8, device=self.device)
        self._sparse_refs = None

    # ------------------------------------------------------------------ state
    def close(self) -> None:
        if getattr(self, "_h", None):
            torch.cuda.synchronize(self.device)
            library().oprag_index_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def n_rows(self) -> int:
        n = ctypes.c_int64()
        _check(library().oprag_index_size(self._h, ctypes.byref(n)))
        return n.value

    def __len__(self) -> int:
        return self.n_rows

    # ------------------------------------------------------------------ upsert
    def upsert(self, rows: torch.Tensor) -> int:
        """Append rows (index dtype, or fp32 for a bf16/fp16 index); returns the first new id."""
        if rows.dtype not in _DTYPE:
            raise OpragError(-1, f"unsupported rows dtype {rows.dtype}")
        if rows.dim() != 2 or rows.shape[1] != self.dim:
            raise OpragError(-1, f"rows must be [m x {self.dim}]")
        _dev_tensor(rows, rows.dtype, self.device, "rows")
        first = ctypes.c_int64()
        _check(library().oprag_upsert(self._h, _ptr(rows) if rows.numel() else None, _DTYPE[rows.dtype],
                                      rows.shape[0], _stream(self.device), ctypes.byref(first)))
        return first.value

    def upsert_pooled(self, hidden: torch.Tensor, lengths: torch.Tensor) -> int:
        """Mean-pool hidden states [m x T x dim] (bf16 or fp32) over each chunk's first lengths[i]
        tokens, L2-normalise, append; returns the first new id."""
        if hidden.dtype not in (torch.bfloat16, torch.float32):
            raise OpragError(-1, f"hidden states must be bf16 or fp32, not {hidden.dtype}")
        if hidden.dim() != 3 or hidden.shape[2] != self.dim:
            raise OpragError(-1, f"hidden must be [m x T x {self.dim}]")
        _dev_tensor(hidden, hidden.dtype, self.device, "hidden")
        _dev_tensor(lengths, torch.int32, self.device, "lengths")
        if lengths.numel() != hidden.shape[0]:
            raise OpragError(-1, "lengths must have m entries")
        first = ctypes.c_int64()
        m = hidden.shape[0]
        _check(library().oprag_upsert_pooled(self._h, _ptr(hidden) if m else None, _DTYPE[hidden.dtype],
                                             _ptr(lengths) if m else None, m, max(1, hidden.shape[1]),
                                             _stream(self.device), ctypes.byref(first)))
        return first.value

    def attach_sparse(self, term_indptr: torch.Tensor, post_chunk: torch.Tensor, post_tf: torch.Tensor,
                      doc_len: torch.Tensor, k1: float = 1.2, b: float = 0.75) -> None:
        """Attach a CSR term -> (chunk, tf) postings index for BM25 (tensors stay referenced)."""
        _dev_tensor(term_indptr, torch.int64, self.device, "term_indptr")
        _dev_tensor(post_chunk, torch.int32, self.device, "post_chunk")
        _dev_tensor(post_tf, torch.int32, self.device, "post_tf")
        _dev_tensor(doc_len, torch.int32, self.device, "doc_len")
        vocab = term_indptr.numel() - 1
        _check(library().oprag_sparse_attach(self._h, vocab, doc_len.numel(), post_chunk.numel(), _ptr(term_indptr),
                                             _ptr(post_chunk), _ptr(post_tf), _ptr(doc_len), k1, b,
                                             _stream(self.device)))
        self._sparse_refs = (term_indptr, post_chunk, post_tf, doc_len)

    # ------------------------------------------------------------------ workspace
    def workspace_bytes(self, op: int, nq: int, k_dense: int = 1, k_sparse: int = 1) -> int:
        n = ctypes.c_size_t()
        _check(library().oprag_workspace_bytes(self._h, op, nq, k_dense, k_sparse, ctypes.byref(n)))
        return n.value

    def workspace(self, op: int, nq: int, k_dense: int = 1, k_sparse: int = 1) -> torch.Tensor:
        """The cached device workspace, grown (never shrunk) to what the call needs."""
        need = self.workspace_bytes(op, nq, k_dense, k_sparse)
        if self._ws.numel() < need:
            self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        return self._ws

    # ------------------------------------------------------------------ search
    def search_dense(self, q: torch.Tensor, k: int, out: tuple | None = None):
        """Exact top-k by inner product. Returns (scores fp32 [nq x k], ids int64 [nq x k])."""
        _dev_tensor(q, self.dtype, self.device, "q")
        nq = q.shape[0]
        scores, ids = out if out is not None else (
            torch.empty((nq, k), dtype=torch.float32, device=self.device),
            torch.empty((nq, k), dtype=torch.int64, device=self.device))
        ws = self.workspace(OP_DENSE, nq, k, 1)
        _check(library().oprag_search_dense(self._h, _ptr(q), nq, k, _ptr(scores), _ptr(ids), _ptr(ws),
                                            ws.numel(), _stream(self.device)))
        return scores, ids

    def search_dense_noalloc(self, q: torch.Tensor, k: int, out: tuple | None = None):
        """search_dense without a workspace: the library's fixed per-GPU scratch array holds the
        intermediate lists (for callers that cannot allocate; concurrent calls on one GPU race)."""
        _dev_tensor(q, self.dtype, self.device, "q")
        nq = q.shape[0]
        scores, ids = out if out is not None else (
            torch.empty((nq, k), dtype=torch.float32, device=self.device),
            torch.empty((nq, k), dtype=torch.int64, device=self.device))
        _check(library().oprag_search_dense_noalloc(self._h, _ptr(q), nq, k, _ptr(scores), _ptr(ids),
                                                    _stream(self.device)))
        return scores, ids

    def search_sparse(self, qterm_indptr: torch.Tensor, qterms: torch.Tensor, k: int, out: tuple | None = None):
        """Exact BM25 top-k. Returns (scores fp32 [nq x k], ids int64 [nq x k])."""
        _dev_tensor(qterm_indptr, torch.int32, self.device, "qterm_indptr")
        _dev_tensor(qterms, torch.int32, self.device, "qterms")
        nq = qterm_indptr.numel() - 1
        scores, ids = out if out is not None else (
            torch.empty((nq, k), dtype=torch.float32, device=self.device),
            torch.empty((nq, k), dtype=torch.int64, device=self.device))
        ws = self.workspace(OP_SPARSE, nq, 1, k)
        _check(library().oprag_search_sparse(self._h, _ptr(qterm_indptr), _ptr(qterms), nq, k, _ptr(scores),
                                             _ptr(ids), _ptr(ws), ws.numel(), _stream(self.device)))
        return scores, ids

    def search_hybrid(self, q: torch.Tensor, qterm_indptr: torch.Tensor, qterms: torch.Tensor, k_dense: int = 100,
                      k_sparse: int = 100, rrf_k: int = 60, k: int = 5, out: tuple | None = None):
        """Dense top-k_dense + BM25 top-k_sparse fused by RRF. Returns (fused fp32, ids int64), [nq x k]."""
        _dev_tensor(q, self.dtype, self.device, "q")
        _dev_tensor(qterm_indptr, torch.int32, self.device, "qterm_indptr")
        _dev_tensor(qterms, torch.int32, self.device, "qterms")
        nq = q.shape[0]
        if qterm_indptr.numel() != nq + 1:
            raise OpragError(-1, "qterm_indptr must have nq + 1 entries")
        fused, ids = out if out is not None else (
            torch.empty((nq, k), dtype=torch.float32, device=self.device),
            torch.empty((nq, k), dtype=torch.int64, device=self.device))
        ws = self.workspace(OP_HYBRID, nq, k_dense, k_sparse)
        _check(library().oprag_search_hybrid(self._h, _ptr(q), nq, _ptr(qterm_indptr), _ptr(qterms), k_dense,
                                             k_sparse, rrf_k, k, _ptr(fused), _ptr(ids), _ptr(ws), ws.numel(),
                                             _stream(self.device)))
        return fused, ids

    def search_hybrid_dense_first(self, q: torch.Tensor, qterm_indptr: torch.Tensor, qterms: torch.Tensor,
                                  n_cand: int = 128, rrf_k: int = 60, k: int = 5, out: tuple | None = None):
        """Dense top-n_cand candidates reranked by BM25 and fused with their dense order by RRF.
        Returns (fused fp32, ids int64), [nq x k]."""
        _dev_tensor(q, self.dtype, self.device, "q")
        _dev_tensor(qterm_indptr, torch.int32, self.device, "qterm_indptr")
        _dev_tensor(qterms, torch.int32, self.device, "qterms")
        nq = q.shape[0]
        if qterm_indptr.numel() != nq + 1:
            raise OpragError(-1, "qterm_indptr must have nq + 1 entries")
        fused, ids = out if out is not None else (
            torch.empty((nq, k), dtype=torch.float32, device=self.device),
            torch.empty((nq, k), dtype=torch.int64, device=self.device))
        ws = self.workspace(OP_DENSE_FIRST, nq, n_cand, 1)
        _check(library().oprag_search_hybrid_dense_first(self._h, _ptr(q), nq, _ptr(qterm_indptr), _ptr(qterms),
                                                         n_cand, rrf_k, k, _ptr(fused), _ptr(ids), _ptr(ws),
                                                         ws.numel(), _stream(self.device)))
        return fused, ids

    def search_hybrid_weighted(self, q: torch.Tensor, qterm_indptr: torch.Tensor, qterms: torch.Tensor,
                               w_dense: float = 0.5, w_lex: float = 0.5, k: int = 5, out: tuple | None = None):
        """w_dense * minmax(dense) + w_lex * minmax(BM25) over every chunk, top k.
        Returns (scores fp32, ids int64), [nq x k]."""
        _dev_tensor(q, self.dtype, self.device, "q")
        _dev_tensor(qterm_indptr, torch.int32, self.device, "qterm_indptr")
        _dev_tensor(qterms, torch.int32, self.device, "qterms")
        nq = q.shape[0]
        if qterm_indptr.numel() != nq + 1:
            raise OpragError(-1, "qterm_indptr must have nq + 1 entries")
        scores, ids = out if out is not None else (
            torch.empty((nq, k), dtype=torch.float32, device=self.device),
            torch.empty((nq, k), dtype=torch.int64, device=self.device))
        ws = self.workspace(OP_WEIGHTED, nq, 1, 1)
        _check(library().oprag_search_hybrid_weighted(self._h, _ptr(q), nq, _ptr(qterm_indptr), _ptr(qterms),
                                                      w_dense, w_lex, k, _ptr(scores), _ptr(ids), _ptr(ws),
                                                      ws.numel(), _stream(self.device)))
        return scores, ids


def rrf_fuse(dense_ids: torch.Tensor, sparse_ids: torch.Tensor, rrf_k: int = 60, k: int = 5):
    """Reciprocal rank fusion of two int64 id lists per query on the GPU. Returns (fused fp32, ids int64)."""
    dev = dense_ids.device
    _dev_tensor(dense_ids, torch.int64, dev, "dense_ids")
    _dev_tensor(sparse_ids, torch.int64, dev, "sparse_ids")
    nq = dense_ids.shape[0]
    if sparse_ids.shape[0] != nq:
        raise OpragError(-1, "both lists need the same number of queries")
    fused = torch.empty((nq, k), dtype=torch.float32, device=dev)
    ids = torch.empty((nq, k), dtype=torch.int64, device=dev)
    _check(library().oprag_rrf_fuse(_ptr(dense_ids), dense_ids.shape[1], _ptr(sparse_ids), sparse_ids.shape[1], nq,
                                    rrf_k, k, _ptr(fused), _ptr(ids), _stream(dev)))
    return fused, ids


def probe_read(src: torch.Tensor, blocks: int, sink: torch.Tensor) -> None:
    """A plain streaming read of all of `src` (contiguous device memory, a multiple of 16
    bytes) in `blocks` workgroups; `sink` (int32, at least `blocks` entries) receives one fold
    per workgroup (oprag_probe_read)."""
    if not (src.is_cuda and src.is_contiguous() and sink.is_cuda and sink.dtype == torch.int32):
        raise OpragError(-1, "src must be contiguous device memory, sink a device int32 tensor")
    if sink.numel() < blocks:
        raise OpragError(-1, "sink holds fewer than blocks entries")
    _check(library().oprag_probe_read(_ptr(src), src.numel() * src.element_size(), blocks, _ptr(sink),
                                      _stream(src.device)))


def time_next_dense_kernel(start: torch.cuda.Event | None, stop: torch.cuda.Event | None) -> None:
    """Arm two timing events that the next dense search from this thread records on its stream
    right before and after its scoring kernel (oprag_time_next_dense_kernel). None, None disarms."""
    if (start is None) != (stop is None):
        raise OpragError(-1, "pass both events or neither")
    a = ctypes.c_void_p(start.cuda_event) if start is not None else None
    b = ctypes.c_void_p(stop.cuda_event) if stop is not None else None
    _check(library().oprag_time_next_dense_kernel(a, b))
