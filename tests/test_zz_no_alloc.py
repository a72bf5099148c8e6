"""The dense search without allocation (a fixed per-GPU scratch array instead of a caller
workspace) against oprag_search_dense, through the C ABI: bit-identical ids and scores on two
calls in a row, the second with a smaller input, and the oracle's acceptance rules."""
import ctypes

import numpy as np
import pytest
import torch

import synth
from tests.gpu_helpers import check_dense, device, log, make_index, oracle_scores

pytestmark = pytest.mark.gpu


def _noalloc(idx, q, k):
    import paper_2608_08340_amd as P
    nq = q.shape[0]
    sc = torch.full((nq, k), 7.0, dtype=torch.float32, device=q.device)
    ids = torch.full((nq, k), -7, dtype=torch.int64, device=q.device)
    st = P.library().oprag_search_dense_noalloc(idx._h, ctypes.c_void_p(q.data_ptr()), nq, k,
                                                ctypes.c_void_p(sc.data_ptr()), ctypes.c_void_p(ids.data_ptr()),
                                                ctypes.c_void_p(torch.cuda.current_stream(q.device).cuda_stream))
    assert st == 0, P.library().oprag_last_error()
    return sc, ids


@pytest.mark.parametrize("dtype,n,d,k,nq1,nq2", [("bf16", 32768, 1024, 5, 256, 16),
                                                 ("bf16", 32768, 1024, 16, 64, 1),
                                                 ("f16", 20000, 384, 100, 40, 7),
                                                 ("f32", 3000, 128, 10, 33, 2)])
def test_noalloc_matches_workspace_search(dtype, n, d, k, nq1, nq2):
    dev = device()
    w = synth.mixture_dense(6100 + k, n, d, 64, nq1, k, dtype)
    idx = make_index(w.rows, dtype)
    for nq in (nq1, nq2):  # the second call smaller: stale lists of the first must not leak in
        log("noalloc", dtype, n, d, k, nq)
        q = w.queries[:nq].contiguous().to(dev)
        s_ref, i_ref = idx.search_dense(q, k)
        s_na, i_na = _noalloc(idx, q, k)
        torch.cuda.synchronize()
        assert torch.equal(i_na, i_ref)
        assert torch.equal(s_na.view(torch.int32), s_ref.view(torch.int32))
        S, X, Q = oracle_scores(w.rows, w.queries[:nq], dtype)
        check_dense(S, X, Q, i_na, s_na, k, dtype, label=f"noalloc nq={nq}")


def test_noalloc_rejects_what_does_not_fit():
    """k > 16 keeps a candidate slot per row below 32,768 rows: 256 queries over 32,768 rows
    need 64 MiB, more than the 32 MiB array, so the call fails before enqueueing anything."""
    import paper_2608_08340_amd as P
    dev = device()
    idx = make_index(torch.zeros((32768, 128), dtype=torch.bfloat16), "bf16")
    q = torch.zeros((256, 128), dtype=torch.bfloat16, device=dev)
    sc = torch.full((256, 100), 7.0, device=dev)
    ids = torch.full((256, 100), -7, dtype=torch.int64, device=dev)
    st = P.library().oprag_search_dense_noalloc(idx._h, ctypes.c_void_p(q.data_ptr()), 256, 100,
                                                ctypes.c_void_p(sc.data_ptr()), ctypes.c_void_p(ids.data_ptr()), None)
    torch.cuda.synchronize()
    assert st == -2, st
    assert (ids == -7).all() and (sc == 7.0).all()
