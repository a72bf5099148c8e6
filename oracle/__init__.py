"""CPU oracle for the OpRAG retrieval hot path.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg import this package;
the library never calls it, and it shares no code, table or helper with the HIP path.

It is the plain definition of what the hot path computes, in fp64 on the exact stored
values, with no blocking, fusion or pruning:

* ``dense``  - retrieval R_k = Op_retrieve(q, I) (Section 3.2, "Retrieval"; Section 4.4):
  inner-product scores of each query against every indexed unit vector, then a full stable
  sort and the first k, ties by ascending row id.
* ``bm25``   - lexical scores with exact full-corpus BM25 semantics (Section 4.4), by a
  document-wise scan of the raw token sequences (no postings index).
* ``rrf``    - reciprocal rank fusion of a dense and a sparse ranked list, in exact rational
  arithmetic (the fusion the hybrid workload specifies; the paper's own weighted fusion of
  Section 4.4 has unstated weights).
* ``upsert`` - append-only Op_upsert (Section 3.2, "Upsert") on a host copy of the index,
  with the fp32 -> bf16 / fp16 rounding the library applies when the source dtype differs.
* ``accept`` - the tie-aware acceptance rules the GPU results are held to.
* ``dense_first``, ``weighted``, ``embed_tail`` - the dense-first hybrid schedule, the
  paper's weighted score fusion and the mean-pool + L2 tail of the embedding step.

Where the paper is silent, each module's docstring states the reading it takes.
"""
from . import accept, bm25, dense, rrf, storage, upsert  # noqa: F401
