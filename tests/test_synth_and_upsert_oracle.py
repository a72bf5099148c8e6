"""Generators are seeded and shaped as stated; the host upsert model is append-only and
all-or-nothing (no GPU)."""
import numpy as np
import pytest

import synth
from oracle.storage import decode, round_f32_to_bf16
from oracle.upsert import HostIndex


def test_seeded_and_deterministic():
    a = synth.mixture_dense(50, 2000, 128, 16, 10, 5, "bf16")
    b = synth.mixture_dense(50, 2000, 128, 16, 10, 5, "bf16")
    assert np.array_equal(synth.storage_bits(a.rows), synth.storage_bits(b.rows))
    assert np.array_equal(synth.storage_bits(a.queries), synth.storage_bits(b.queries))
    c = synth.mixture_dense(51, 2000, 128, 16, 10, 5, "bf16")
    assert not np.array_equal(synth.storage_bits(a.rows), synth.storage_bits(c.rows))


def test_chunked_draw_is_thread_count_independent():
    cen = synth.mixture_centres(synth.rng(60, 0), 8, 64)
    x1 = synth.mixture_rows_chunked(60, 1, cen, 3000, 0.3, chunk=512, threads=1)
    x4 = synth.mixture_rows_chunked(60, 1, cen, 3000, 0.3, chunk=512, threads=4)
    assert np.array_equal(x1, x4)


def test_shapes_norms_and_rounding():
    w = synth.tiny_dense()
    assert tuple(w.rows.shape) == (1024, 384) and tuple(w.queries.shape) == (16, 384)
    n = np.linalg.norm(synth.upcast_f32(w.rows).astype(np.float64), axis=1)
    assert np.abs(n - 1).max() < 1e-5
    x = synth.mixture_rows(synth.rng(61, 1), synth.mixture_centres(synth.rng(61, 0), 4, 256), 100, 0.3)
    assert np.array_equal(synth.storage_bits(synth.to_storage(x, "bf16")), round_f32_to_bf16(x))


def test_sparse_corpus_moments():
    ind, toks = synth.sparse_corpus(synth.rng(62, 3), 4096, 30000, 1.1, 256.0)
    lens = np.diff(ind)
    assert abs(lens.mean() - 256) < 2 and abs(lens.var() - 256) < 40
    p = synth.zipf_pmf(30000, 1.1)
    freq = np.bincount(toks, minlength=30000) / toks.shape[0]
    assert abs(freq[0] - p[0]) < 0.01 and abs(freq[1] / freq[0] - 2 ** -1.1) < 0.02
    qi, qt = synth.zipf_query_terms(synth.rng(62, 4), 64, 8, 30000, 1.1)
    assert qi[-1] == 512 and qt.min() >= 0 and qt.max() < 30000


def test_host_upsert_model():
    h = HostIndex(4, 5, "bf16")
    x = np.arange(12, dtype=np.float32).reshape(3, 4) / 7
    assert h.append_f32(x) == 0 and h.n_rows == 3
    before = h.bits.copy()
    with pytest.raises(OverflowError):
        h.append_f32(np.ones((3, 4), np.float32))
    assert h.n_rows == 3 and np.array_equal(h.bits, before)
    assert h.append_bits(round_f32_to_bf16(np.ones((2, 4), np.float32))) == 3
    assert np.array_equal(decode(h.valid_bits()[3:], "bf16"), np.ones((2, 4)))
