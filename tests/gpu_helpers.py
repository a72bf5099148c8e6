"""Helpers shared by the GPU parity tests (not a test module)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import synth
from oracle import accept
from oracle import dense as od
from oracle.storage import decode

DT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
RTOL = {"f32": 1e-5, "bf16": 2e-3, "f16": 2e-3}


def device() -> torch.device:
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_08340_amd as P

    P.library()  # fails loudly when the HIP library is missing
    return torch.device("cuda", 0)


def log(*a) -> None:
    print(*a, flush=True, file=sys.stderr)


def make_index(rows: torch.Tensor, dtype: str, capacity: int | None = None):
    from paper_2608_08340_amd import Index

    dev = device()
    n, d = rows.shape
    idx = Index(d, capacity or max(n, 1), DT[dtype])
    if n:
        idx.upsert(rows.to(dev))
    return idx


def oracle_scores(rows: torch.Tensor, queries: torch.Tensor, dtype: str):
    X = decode(synth.storage_bits(rows), dtype)
    Q = decode(synth.storage_bits(queries), dtype)
    return od.scores(X, Q), X, Q


def check_dense(S, X, Q, ids, scores, k, dtype, strict=True, label=""):
    """Both acceptance modes over every query; raises with the first problems."""
    ids = ids.cpu().numpy() if isinstance(ids, torch.Tensor) else ids
    scores = scores.cpu().numpy() if isinstance(scores, torch.Tensor) else scores
    reps = accept.check_batch(S, ids, scores, k, rtol=RTOL[dtype])
    bad = [(q, r.problems) for q, r in enumerate(reps) if not r.ok]
    assert not bad, f"{label} rel mode: {len(bad)} queries fail, first: {bad[:2]}"
    if strict:
        E = accept.strict_err(od.abs_dot(X, Q), X.shape[1])
        reps = accept.check_batch(S, ids, scores, k, mode="strict", err=E)
        bad = [(q, r.problems) for q, r in enumerate(reps) if not r.ok]
        assert not bad, f"{label} strict mode: {len(bad)} queries fail, first: {bad[:2]}"
    return reps
