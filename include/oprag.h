/*
 * oprag.h - C ABI of the MI355X (gfx950) exact-retrieval core of OpRAG.
 *
 * The paper's operator model (Section 3.2) states the three calls this library implements:
 *   E  = Op_embed(D; b_e)          - the model forward pass is outside the library; its tail
 *                                    (mean pool, L2 normalisation, Section 4.3) is fused with
 *                                    the insertion in oprag_upsert_pooled, and oprag_upsert
 *                                    takes vectors that are already unit-norm;
 *   I' = Op_upsert(I, E; b_u)      - oprag_upsert: bulk insertion of new embeddings;
 *   R_k = Op_retrieve(q, I)        - oprag_search_dense: exact top-k by inner product;
 * and the hybrid retrieval of Section 4.4 (dense scores plus inverted-postings BM25 over the
 * full corpus, fused, then partial top-k): oprag_sparse_attach / oprag_search_sparse /
 * oprag_rrf_fuse / oprag_search_hybrid (reciprocal rank fusion) and
 * oprag_search_hybrid_weighted (the paper's weighted score fusion), plus the dense-first
 * serving schedule of Sections 4.1 and 5.5, oprag_search_hybrid_dense_first.
 *
 * Conventions for every function:
 *  - Return value: OPRAG_OK (0) or a negative oprag_status; the reason is available from
 *    oprag_last_error() (thread-local string).  Nothing throws across the ABI.
 *  - Validation is synchronous and complete before anything is enqueued: on error nothing
 *    is enqueued and the index is unchanged.  Faults inside kernels surface at the caller's
 *    next synchronisation of the stream.
 *  - Memory: every large buffer (slab, CSR arrays, queries, outputs, workspace) is device
 *    memory owned by the caller and must stay valid while the index or call uses it.  The
 *    library allocates only its BM25 arrays at attach time (8 bytes per term, 12 per posting,
 *    8 per chunk and at most 64 MiB of dense rows for the most frequent terms, plus temporary
 *    counters) and never in create, upsert or search.
 *    Device pointers must be 16-byte aligned.
 *  - Streams: `stream` is a hipStream_t (NULL = default stream).  Calls are asynchronous on
 *    it.  An index keeps host-side state (row count), so calls on one index must be issued
 *    from one host thread at a time; an upsert is seen by searches ordered after it on the
 *    device (same stream, or ordered by the caller with events).  A workspace holds
 *    intermediate results of one call: concurrent calls need separate workspaces.
 *  - Ranked lists are ordered by score descending, then id ascending.  Lists shorter than k
 *    are padded with id -1 and score -inf.  1 <= k <= OPRAG_MAX_K.
 */
#ifndef OPRAG_H_
#define OPRAG_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OPRAG_ABI_VERSION 2
#define OPRAG_MAX_K 128
#define OPRAG_MAX_DIM 8192

typedef enum oprag_status {
  OPRAG_OK = 0,
  OPRAG_E_INVALID = -1,     /* bad argument (null/misaligned pointer, size, dtype, k, ...) */
  OPRAG_E_CAPACITY = -2,    /* upsert would exceed the slab capacity */
  OPRAG_E_STATE = -3,       /* call not valid in the index's state (e.g. no sparse index) */
  OPRAG_E_UNSUPPORTED = -4, /* valid request outside what this build supports */
  OPRAG_E_DEVICE = -5       /* a HIP call failed */
} oprag_status;

typedef enum oprag_dtype { OPRAG_F32 = 0, OPRAG_BF16 = 1, OPRAG_F16 = 2 } oprag_dtype;

typedef enum oprag_op {
  OPRAG_OP_DENSE = 0,
  OPRAG_OP_SPARSE = 1,
  OPRAG_OP_HYBRID = 2,
  OPRAG_OP_DENSE_FIRST = 3,
  OPRAG_OP_WEIGHTED = 4
} oprag_op;

typedef struct oprag_index oprag_index; /* opaque handle */

typedef struct oprag_index_desc {
  int32_t dim;      /* vector dimension d: 1..OPRAG_MAX_DIM; multiple of 4 (f32) or 128 (bf16, f16) */
  int32_t dtype;    /* oprag_dtype of the stored vectors and of queries */
  int64_t capacity; /* rows the slab holds: 1 .. 2^31 - 2 */
  int32_t device;   /* HIP device ordinal of the slab */
  int32_t reserved; /* must be 0 */
} oprag_index_desc;

int32_t oprag_abi_version(void);

/* Message describing the last failure on this thread ("" if none). */
const char *oprag_last_error(void);

/*
 * Create an index over a caller-owned slab: row-major [capacity x dim] in desc->dtype,
 * slab_bytes >= capacity * dim * sizeof(dtype).  The index starts empty (n_rows = 0);
 * row ids are insertion positions.  Allocates nothing on the device.
 * Errors: E_INVALID (desc, slab, out, device ordinal), E_DEVICE.
 */
oprag_status oprag_index_create(const oprag_index_desc *desc, void *slab_dev, size_t slab_bytes, oprag_index **out);

/* Release the handle and the arrays the library allocated; never touches caller buffers.
 * The caller must make sure no work using the index is still pending.  NULL is OK. */
oprag_status oprag_index_destroy(oprag_index *idx);

/* Rows currently in the index (host state, advanced when an upsert is enqueued). */
oprag_status oprag_index_size(const oprag_index *idx, int64_t *n_rows);

/*
 * Upsert (Section 3.2, "Upsert"; bulk commit, Section 4.1), append-only: copies m rows
 * [m x dim] of rows_dtype into slab rows [n_rows, n_rows + m) and advances n_rows.
 * rows_dtype must equal the index dtype, or be OPRAG_F32 for a bf16 / f16 index (converted
 * with round-to-nearest-even).  All or nothing: if n_rows + m > capacity nothing is
 * enqueued and E_CAPACITY is returned.  m = 0 is a no-op.  *first_row (may be NULL)
 * receives the id of the first new row.  Searches enqueued later on the same stream see
 * the new rows.
 */
oprag_status oprag_upsert(oprag_index *idx, const void *rows_dev, int32_t rows_dtype, int64_t m, void *stream,
                          int64_t *first_row);

/*
 * Embedding tail fused with the upsert: Op_embed's last two steps (Section 4.3: mean pool of
 * the model's hidden states over the chunk's tokens, then L2 normalisation) followed by
 * Op_upsert of the resulting vectors (appended as in oprag_upsert, all or nothing).
 *   hidden_dev  [m x T x dim] in hidden_dtype (OPRAG_BF16 or OPRAG_F32), chunk-major;
 *   lengths_dev [m] int32: chunk i's tokens are 0 .. lengths[i] - 1 (right padding; values
 *               outside [0, T] are clamped).
 * Row n_rows + i becomes sum / ||sum|| of chunk i's valid hidden states (sums in fp32 in token
 * order, the norm in fp64; the mean's 1/len cancels), rounded to nearest even to the index
 * dtype; a chunk with no tokens or a zero sum becomes the zero vector.  *first_row (optional)
 * receives the first new id.  Asynchronous on `stream`.
 */
oprag_status oprag_upsert_pooled(oprag_index *idx, const void *hidden_dev, int32_t hidden_dtype,
                                 const int32_t *lengths_dev, int64_t m, int32_t T, void *stream, int64_t *first_row);

/*
 * Attach the inverted-postings index BM25 scores from (Section 4.4): CSR term -> (chunk, tf)
 * over chunk ids [0, n_docs) (the same ids as the dense rows; n_docs <= capacity).
 *   term_indptr_dev [vocab + 1] int64, term_indptr[0] = 0, term_indptr[vocab] = nnz;
 *   post_chunk_dev  [nnz] int32, strictly ascending within a term, in [0, n_docs);
 *   post_tf_dev     [nnz] int32 >= 1;  doc_len_dev [n_docs] int32 >= 0 (tokens per chunk).
 * The arrays stay caller-owned and are read by later searches.  The library checks them on
 * the device (E_INVALID on any violation), then computes idf(t) = ln(1 + (N - df + 0.5) /
 * (df + 0.5)) per term and tf / (tf + k1 (1 - b + b dl / avgdl)) per posting, in fp64 stored
 * as fp32, a chunk-major copy of (term, weight) pairs for scoring given chunks, and dense
 * per-chunk weight rows of the most frequent terms (df >= max(64, n_docs / 8), at most 992 rows
 * and 64 MiB), into arrays it owns (8 bytes per term, 12 per posting, 8 per chunk, plus the
 * rows).
 * Synchronises `stream`.  Re-attaching replaces the previous sparse index.
 * k1 >= 0, 0 <= b <= 1.
 */
oprag_status oprag_sparse_attach(oprag_index *idx, int32_t vocab, int64_t n_docs, int64_t nnz,
                                 const int64_t *term_indptr_dev, const int32_t *post_chunk_dev,
                                 const int32_t *post_tf_dev, const int32_t *doc_len_dev, float k1, float b,
                                 void *stream);

/*
 * Workspace bytes a search of nq queries needs (op: oprag_op; k_dense is the dense k for
 * OPRAG_OP_DENSE and OPRAG_OP_HYBRID and the candidate count n_cand for
 * OPRAG_OP_DENSE_FIRST, k_sparse the sparse k for OPRAG_OP_SPARSE and OPRAG_OP_HYBRID).  The value does not depend on the current row count, so a workspace
 * sized once stays valid as the index grows.
 */
oprag_status oprag_workspace_bytes(const oprag_index *idx, int32_t op, int64_t nq, int32_t k_dense, int32_t k_sparse,
                                   size_t *bytes);

/*
 * Exact dense top-k, R_k = Op_retrieve(q, I) (Section 3.2, "Retrieval"; scoring by matrix
 * products over the embedding matrix and partial top-k selection, Section 4.4):
 * s(q, i) = sum_j Q[q, j] X[i, j] over rows 0 <= i < n_rows, accumulated in fp32.
 *   q_dev      [nq x dim] in the index dtype;
 *   scores_dev [nq x k] fp32;  ids_dev [nq x k] int64 (row ids).
 * nq = 0 is a no-op.  workspace_dev must hold oprag_workspace_bytes(OPRAG_OP_DENSE) bytes.
 * Asynchronous on stream for every k (bf16 / fp16 searches with k > 16 run in threshold
 * levels whose exactness repair is decided on the device), so a search can be captured in a
 * HIP graph.
 */
oprag_status oprag_search_dense(const oprag_index *idx, const void *q_dev, int64_t nq, int32_t k, float *scores_dev,
                                int64_t *ids_dev, void *workspace_dev, size_t workspace_bytes, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): oprag_search_dense with the same
 * arguments, kernels and results, but no workspace argument.  The intermediate per-chunk
 * lists (or threshold-level candidates) go to a fixed array of OPRAG_NOALLOC_SCRATCH_BYTES
 * in device memory that the library defines once per GPU and keeps until the process ends;
 * the call allocates nothing.  A search whose plan at the current row count needs more
 * returns E_CAPACITY with nothing enqueued: split the batch.  The need never exceeds what
 * oprag_workspace_bytes(OPRAG_OP_DENSE) reports; with k <= 16 and up to 1,024 queries it
 * stays within 8 MiB (2.6 MB for 256 queries and k = 5), while k > 16 needs 8 bytes per
 * query and candidate slot (every row up to 32,768 rows) and can exceed the array at a few
 * hundred queries.  Every call on one GPU shares its array, and nothing in it has to start
 * at any value (each call writes what it later reads), so calls that may overlap on one GPU
 * (different streams, or several host threads) race and must be ordered by the caller.
 */
#define OPRAG_NOALLOC_SCRATCH_BYTES (32u << 20)
oprag_status oprag_search_dense_noalloc(const oprag_index *idx, const void *q_dev, int64_t nq, int32_t k,
                                        float *scores_dev, int64_t *ids_dev, void *stream);

/*
 * Exact BM25 top-k (Section 4.4) over the attached sparse index.  Query q's terms are
 * qterms_dev[qterm_indptr_dev[q] .. qterm_indptr_dev[q + 1]) (int32; repeated terms count
 * once per occurrence; ids outside [0, vocab) match nothing).  Only chunks with a positive
 * score are ranked.  scores_dev [nq x k] fp32, ids_dev [nq x k] int64.
 * E_STATE without an attached sparse index.
 */
oprag_status oprag_search_sparse(const oprag_index *idx, const int32_t *qterm_indptr_dev, const int32_t *qterms_dev,
                                 int64_t nq, int32_t k, float *scores_dev, int64_t *ids_dev, void *workspace_dev,
                                 size_t workspace_bytes, void *stream);

/*
 * Reciprocal rank fusion of two ranked id lists per query (the fusion the hybrid workload
 * specifies; the paper's own Section 4.4 fusion is a weighted score sum with unstated
 * weights): fused(d) = sum over lists holding d of 1 / (rrf_k + rank), ranks 1-based over
 * the list's valid prefix (ids >= 0; ids within one list are distinct, as search outputs are).
 * Compared exactly as rationals; ties by ascending id.
 *   dense_ids_dev [nq x k_dense] int64, sparse_ids_dev [nq x k_sparse] int64;
 *   fused_dev [nq x k] fp32 (the exact value rounded to fp32), ids_dev [nq x k] int64.
 * 0 <= rrf_k <= 1000000.  Needs no index and no workspace.
 */
oprag_status oprag_rrf_fuse(const int64_t *dense_ids_dev, int32_t k_dense, const int64_t *sparse_ids_dev,
                            int32_t k_sparse, int64_t nq, int32_t rrf_k, int32_t k, float *fused_dev,
                            int64_t *ids_dev, void *stream);

/*
 * Hybrid search (Section 4.4): exact dense top-k_dense and exact BM25 top-k_sparse over the
 * full corpus, fused by reciprocal rank fusion (rrf_k), cut at k.  Equivalent to
 * oprag_search_dense + oprag_search_sparse + oprag_rrf_fuse on the same stream.
 * workspace_dev must hold oprag_workspace_bytes(OPRAG_OP_HYBRID) bytes.
 */
oprag_status oprag_search_hybrid(const oprag_index *idx, const void *q_dev, int64_t nq, const int32_t *qterm_indptr_dev,
                                 const int32_t *qterms_dev, int32_t k_dense, int32_t k_sparse, int32_t rrf_k, int32_t k,
                                 float *fused_dev, int64_t *ids_dev, void *workspace_dev, size_t workspace_bytes,
                                 void *stream);

/*
 * Dense-first hybrid search (the serving schedule of Section 4.1, "Retrieval", whose latency
 * and quality against full hybrid retrieval Section 5.5 reports): the exact dense top-n_cand
 * candidates (as oprag_search_dense), their BM25 scores over the attached sparse index (the
 * full-corpus statistics of oprag_sparse_attach; a candidate's terms are read from the
 * chunk-major copy the attach builds), and reciprocal rank fusion (rrf_k) of the candidates' dense order with their
 * lexical order (the candidates with a positive score, by score desc then id asc), cut at k
 * by (fused desc, id asc) and compared exactly as in oprag_rrf_fuse.  Only candidates can be
 * returned.
 *   q_dev [nq x dim]; qterm_indptr_dev / qterms_dev as in oprag_search_sparse;
 *   fused_dev [nq x k] fp32, ids_dev [nq x k] int64 (-1 / -inf past the candidates).
 * 1 <= n_cand <= 128.  workspace_dev must hold
 * oprag_workspace_bytes(OPRAG_OP_DENSE_FIRST, k_dense = n_cand) bytes.  E_STATE without an
 * attached sparse index.
 */
oprag_status oprag_search_hybrid_dense_first(const oprag_index *idx, const void *q_dev, int64_t nq,
                                             const int32_t *qterm_indptr_dev, const int32_t *qterms_dev, int32_t n_cand,
                                             int32_t rrf_k, int32_t k, float *fused_dev, int64_t *ids_dev,
                                             void *workspace_dev, size_t workspace_bytes, void *stream);

/*
 * Weighted score fusion over the whole corpus (Section 4.4): score(d, q) = w_dense *
 * s^_dense(d, q) + w_lex * s^_lexical(d, q) for every chunk 0 <= d < n_rows, where s^ is the
 * per-query min-max normalisation over all chunks, (s - min) / (max - min), and 0 for every
 * chunk when max == min (the paper states the formula but neither s^ nor the weights).
 * s_dense is the inner product (fp32 accumulation), s_lexical the BM25 score of the attached
 * sparse index (0 for chunks without a matching term and for chunks past its n_docs).  The
 * weighted sum is formed in fp64 and rounded to fp32; top k by (score desc, id asc).
 *   q_dev [nq x dim] (bf16 / fp16 index); qterm_indptr_dev / qterms_dev as in
 *   oprag_search_sparse; scores_dev [nq x k] fp32, ids_dev [nq x k] int64.
 * w_dense, w_lex finite and >= 0.  The scores of every chunk pass through the workspace
 * (oprag_workspace_bytes(OPRAG_OP_WEIGHTED): 16 bytes per query and unit of capacity, plus
 * 8 bytes per query for each partial minimum / maximum pair of the two score dumps).
 * E_STATE without an attached sparse index, E_UNSUPPORTED for an fp32 index.
 */
oprag_status oprag_search_hybrid_weighted(const oprag_index *idx, const void *q_dev, int64_t nq,
                                          const int32_t *qterm_indptr_dev, const int32_t *qterms_dev, float w_dense,
                                          float w_lex, int32_t k, float *scores_dev, int64_t *ids_dev,
                                          void *workspace_dev, size_t workspace_bytes, void *stream);

/*
 * Kernel timing (diagnostics: measuring the scoring kernel against its roofline).  Arms a
 * pair of caller-created HIP events (hipEvent_t passed as void *) that the next dense
 * search issued from the calling thread records on its stream immediately before and after
 * its scoring kernel, the kernel that streams the index (the merge of per-chunk lists that
 * may follow stays outside the pair; with more than 2^20 queries only the first launch is
 * bracketed).  One-shot: the pair is disarmed once recorded.  NULL, NULL disarms.  The
 * library creates, keeps and destroys no event.
 */
oprag_status oprag_time_next_dense_kernel(void *start_event, void *stop_event);

/*
 * Read-bandwidth probe (diagnostics: the HBM read rate a plain stream reaches, the ceiling a
 * search's cold pass over the index is compared with).  Reads `bytes` (a positive multiple of
 * 16) from `src_dev` (16-byte aligned, device memory of at least `bytes`) with 16-byte loads,
 * eight in flight per thread, in `blocks` workgroups of 256 threads (1 .. 4,096), grid-
 * strided, and writes one 32-bit fold of the data per workgroup to `sink_dev[0 .. blocks)`
 * (device memory, 16-byte aligned, caller-owned).  Asynchronous on `stream`; E_INVALID for a
 * bad argument.
 */
#define OPRAG_PROBE_MAX_BLOCKS 4096
oprag_status oprag_probe_read(const void *src_dev, size_t bytes, int32_t blocks, uint32_t *sink_dev, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* OPRAG_H_ */
