"""The C-ABI library loads, exports every function include/oprag.h declares, and rejects bad
arguments before touching the device (no GPU needed: no call here reaches a kernel)."""
import ctypes
import os
import re

import pytest

import paper_2608_08340_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oprag.h")

E_INVALID, E_CAPACITY, E_STATE, E_UNSUPPORTED, E_DEVICE = -1, -2, -3, -4, -5


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(oprag_[a-z_]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(P.LIB_PATH):
        pytest.skip("liboprag.so not built")
    return P.library()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(P._SIGS), "binding and header disagree"
    assert lib.oprag_abi_version() == 2


def _desc(dim=1024, dtype=1, cap=100, dev=0, res=0):
    return P._Desc(dim, dtype, cap, dev, res)


@pytest.mark.parametrize("desc,slab,nbytes,why", [
    (_desc(dtype=7), 4096, 1 << 30, "dtype"),
    (_desc(dim=0), 4096, 1 << 30, "dim"),
    (_desc(dim=9000), 4096, 1 << 30, "dim max"),
    (_desc(cap=0), 4096, 1 << 30, "capacity"),
    (_desc(cap=1 << 31), 4096, 1 << 40, "capacity max"),
    (_desc(dev=-1), 4096, 1 << 30, "device"),
    (_desc(res=1), 4096, 1 << 30, "reserved"),
    (_desc(), None, 1 << 30, "null slab"),
    (_desc(), 4097, 1 << 30, "misaligned slab"),
    (_desc(), 4096, 100 * 1024 * 2 - 1, "slab too small"),
])
def test_create_rejects(lib, desc, slab, nbytes, why):
    h = ctypes.c_void_p()
    st = lib.oprag_index_create(ctypes.byref(desc), None if slab is None else ctypes.c_void_p(slab), nbytes,
                                ctypes.byref(h))
    assert st == E_INVALID, why
    assert h.value is None
    assert lib.oprag_last_error()


def test_create_unsupported_dims(lib):
    h = ctypes.c_void_p()
    assert lib.oprag_index_create(ctypes.byref(_desc(dim=100, dtype=1)), ctypes.c_void_p(4096), 1 << 30,
                                  ctypes.byref(h)) == E_UNSUPPORTED
    assert lib.oprag_index_create(ctypes.byref(_desc(dim=64, dtype=2)), ctypes.c_void_p(4096), 1 << 30,
                                  ctypes.byref(h)) == E_UNSUPPORTED
    assert lib.oprag_index_create(ctypes.byref(_desc(dim=6, dtype=0)), ctypes.c_void_p(4096), 1 << 30,
                                  ctypes.byref(h)) == E_UNSUPPORTED
    assert lib.oprag_index_create(None, ctypes.c_void_p(4096), 1 << 30, ctypes.byref(h)) == E_INVALID


def test_valid_create_reaches_device_only_after_validation(lib):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present; covered by the GPU tests")
    h = ctypes.c_void_p()
    st = lib.oprag_index_create(ctypes.byref(_desc()), ctypes.c_void_p(4096), 1 << 30, ctypes.byref(h))
    assert st == E_DEVICE and h.value is None


def test_null_handle_everywhere(lib):
    n = ctypes.c_int64()
    sz = ctypes.c_size_t()
    assert lib.oprag_index_size(None, ctypes.byref(n)) == E_INVALID
    assert lib.oprag_upsert(None, None, 1, 0, None, None) == E_INVALID
    assert lib.oprag_sparse_attach(None, 1, 1, 0, None, None, None, None, 1.2, 0.75, None) == E_INVALID
    assert lib.oprag_workspace_bytes(None, 0, 1, 5, 5, ctypes.byref(sz)) == E_INVALID
    assert lib.oprag_search_dense(None, None, 1, 5, None, None, None, 0, None) == E_INVALID
    assert lib.oprag_search_sparse(None, None, None, 1, 5, None, None, None, 0, None) == E_INVALID
    assert lib.oprag_search_hybrid(None, None, 1, None, None, 100, 100, 60, 5, None, None, None, 0, None) == E_INVALID
    assert lib.oprag_index_destroy(None) == 0


@pytest.mark.parametrize("kd,ks,nq,rk,k,ptr,why", [
    (0, 5, 1, 60, 5, 4096, "k_dense 0"),
    (5, 129, 1, 60, 5, 4096, "k_sparse > 128"),
    (5, 5, 1, 60, 0, 4096, "k 0"),
    (5, 5, 1, -1, 5, 4096, "rrf_k < 0"),
    (5, 5, 1, 1000001, 5, 4096, "rrf_k too big"),
    (5, 5, -1, 60, 5, 4096, "nq < 0"),
    (5, 5, 1, 60, 5, None, "null pointers"),
    (5, 5, 1, 60, 5, 4100, "misaligned"),
])
def test_rrf_rejects(lib, kd, ks, nq, rk, k, ptr, why):
    p = None if ptr is None else ctypes.c_void_p(ptr)
    assert lib.oprag_rrf_fuse(p, kd, p, ks, nq, rk, k, p, p, None) == E_INVALID, why


def test_time_hook_arms_and_disarms(lib):
    assert lib.oprag_time_next_dense_kernel(None, None) == 0
    assert lib.oprag_time_next_dense_kernel(ctypes.c_void_p(4096), None) == E_INVALID
    assert lib.oprag_time_next_dense_kernel(None, ctypes.c_void_p(4096)) == E_INVALID
    assert lib.oprag_time_next_dense_kernel(ctypes.c_void_p(4096), ctypes.c_void_p(8192)) == 0
    assert lib.oprag_time_next_dense_kernel(None, None) == 0  # disarm: nothing is recorded


@pytest.mark.parametrize("src,nbytes,blocks,sink,why", [
    (None, 4096, 4, 4096, "null src"),
    (4096, 4096, 4, None, "null sink"),
    (4096, 0, 4, 4096, "zero bytes"),
    (4096, 4100, 4, 4096, "bytes not a multiple of 16"),
    (4096, 4096, 0, 4096, "no workgroups"),
    (4096, 4096, 4097, 4096, "too many workgroups"),
    (4104, 4096, 4, 4096, "misaligned src"),
])
def test_probe_read_rejects(lib, src, nbytes, blocks, sink, why):
    p = lambda v: None if v is None else ctypes.c_void_p(v)
    assert lib.oprag_probe_read(p(src), nbytes, blocks, p(sink), None) == E_INVALID, why


def test_rrf_empty_batch_is_noop(lib):
    assert lib.oprag_rrf_fuse(None, 5, None, 5, 0, 60, 5, None, None, None) == 0


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(P, "_lib", None)
    monkeypatch.setattr(P, "LIB_PATH", "/nonexistent/liboprag.so")
    with pytest.raises(P.OpragError):
        P.library()
