// Internal declarations shared by the host runtime (api.cpp) and the HIP kernels.
// Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace oprag {

constexpr int kMaxK = 128;                 // largest k any list may ask for
constexpr int kMaxQPerLaunch = 1 << 20;    // queries per dense launch (the host splits larger batches)
constexpr int kDtypeF32 = 0, kDtypeBF16 = 1, kDtypeF16 = 2;

struct DenseArgs {
  const void* X;                // slab rows [n_rows x d]
  long long n_rows;
  int d;
  const void* Q;                // queries of this launch [nq x d]
  int nq;
  int k;
  int n_qblocks;
  int n_chunks;
  long long rows_per_chunk;     // multiple of the kernel's tile rows
  unsigned long long* partial;  // [nq x n_chunks x k] per-chunk lists (when n_chunks > 1)
  float* out_scores;            // [nq x k]
  long long* out_ids;           // [nq x k]
  // Filtered mode (k > 16): every row scoring >= th[q * th_stride] (all rows when th is null)
  // becomes a candidate key in cbuf[q][0 .. cap); ccnt[q] counts them (and may exceed cap).
  const float* th = nullptr;
  int th_stride = 0;
  unsigned long long* cbuf = nullptr;
  int* ccnt = nullptr;
  long long cap = 0;
  // When set, the launch does nothing unless *gate != 0 (a device-side overflow flag).
  const int* gate = nullptr;
  // Score dump (SEL 3): every score to dump[q * dump_ld + row]; with dump_mm set, also the
  // minimum and maximum of each (query, chunk) to dump_mm[(q * n_chunks + chunk) * 2 + {0, 1}].
  float* dump = nullptr;
  long long dump_ld = 0;
  float* dump_mm = nullptr;
};

struct DensePlan {
  int n_cus = 0;                // compute units of the device the plan is for
  int kernel = 0;               // index into the dense kernel table
  int bn = 0;                   // queries per workgroup
  int tile_rows = 0;            // rows per tile
  int n_qblocks = 0;
  int n_chunks = 0;
  long long rows_per_chunk = 0;
  long long cap = 0;            // partial-list slots per query (bounds n_chunks * k)
  long long grid = 0;
  size_t lds_bytes = 0;
  // Filtered mode: candidate passes over growing row prefixes, each one's k-th score the next
  // one's threshold; the last level is all rows.
  bool filtered = false;
  int n_levels = 0;
  long long level_rows[8] = {};
  long long fcap = 0;           // candidate slots per query
  bool repair = false;          // a level can overflow fcap: enqueue the device-gated repair
  long long chunk_bound = 0;    // workgroups per query block the filter passes aim for
  // The first level's kernel: a small-tile one when the main kernel would leave most CUs idle
  // on the first level's few rows.
  int kernel0 = 0;
  int n_qblocks0 = 0;
  long long chunk_bound0 = 0;
};

DensePlan plan_dense(int dtype, int d, long long n_rows, int nq, int k, int n_cus);
// The per-chunk-list plan for any k (the exact fallback of the filtered mode).
DensePlan plan_dense_lists(int dtype, int d, long long n_rows, int nq, int k, int n_cus);
size_t dense_workspace_bytes(const DensePlan& p, int nq);
// Score dump: every score of nq queries against rows [0, a.n_rows) into a.dump (SEL 3 kernel).
DensePlan plan_dense_dump(int dtype, int d, long long n_rows, int nq, int n_cus);
hipError_t launch_dense_dump(const DensePlan& p, const DenseArgs& a, hipStream_t s);
// Weighted fusion of dense scores D and lexical scores B ([nq x ld], lexical 0 past n_lex),
// min-max normalised per query over n chunks, then the exact top k (cbuf [nq x n], ccnt [nq]).
// The minima and maxima come from the dumps' partials mm_d [nq x pd x 2] and mm_l [nq x pl x 2].
hipError_t launch_weighted_fuse(int n_cus, const float* D, const float* B, long long ld, long long n, long long n_lex, int nq,
                                const float* mm_d, int pd, const float* mm_l, int pl, double wd, double wl, int k,
                                unsigned long long* cbuf, int* ccnt, float* out_scores, long long* out_ids,
                                hipStream_t s);
// Plans take the compute-unit count of the index's device (the grid aims at a multiple of it).
// Enough workspace for a search of nq queries at any row count up to `capacity`.
size_t dense_workspace_bound(int dtype, int d, long long capacity, int nq, int k, int n_cus);
// ev0 / ev1 (optional) are recorded on s right before and after the scoring kernel (in
// filtered mode, the last level's).  Filtered mode also enqueues its exactness repair:
// launches gated on device-side overflow flags, so the search never waits for the host.
hipError_t launch_dense(const DensePlan& p, int dtype, const DenseArgs& a, hipStream_t s, hipEvent_t ev0 = nullptr,
                        hipEvent_t ev1 = nullptr);

// ---------------------------------------------------------------- sparse (BM25)
struct SparseIndex {
  int vocab = 0;
  long long n_docs = 0;
  long long nnz = 0;
  const long long* term_indptr = nullptr;   // caller-owned
  const int* post_chunk = nullptr;          // caller-owned
  const int* post_tf = nullptr;             // caller-owned
  float* idfk = nullptr;                    // library-owned [vocab]: idf(t) * (k1 + 1)
  float* wpost = nullptr;                   // library-owned [nnz]: tf / (tf + k1 (1 - b + b dl / avgdl))
  // library-owned chunk-major copy: chunk d's (term, weight) pairs at [fwd_ptr[d], fwd_ptr[d + 1])
  long long* fwd_ptr = nullptr;             // [n_docs + 1]
  int* fwd_term = nullptr;                  // [nnz]
  float* fwd_w = nullptr;                   // [nnz]
  // library-owned dense rows of the head terms (the most frequent ones): row hidx[t] of whead
  // holds term t's posting weight for every chunk, 0 where t is absent
  int n_head = 0;
  long long head_ld = 0;                    // row stride: n_docs rounded up to 4
  int* hidx = nullptr;                      // [vocab]: row of term t, -1 for the other terms
  float* whead = nullptr;                   // [n_head x head_ld]
  double avgdl = 0.0;
  float k1 = 0.f, b = 0.f;
};

constexpr int kSparseRange = 32768;        // chunks scored per workgroup (LDS accumulator, 128 KiB)
constexpr int kMaxHead = 992;              // head terms at most (the kernel lists a query's in LDS)
constexpr long long kHeadBytes = 64ll << 20;  // dense head rows at most

// Validates the CSR on the device; returns the number of violations found (synchronous).
hipError_t sparse_validate(int vocab, long long n_docs, long long nnz, const long long* indptr,
                           const int* chunk, const int* tf, const int* doc_len, unsigned int* d_flag,
                           hipStream_t s);
hipError_t sparse_prepare(SparseIndex& sp, const int* doc_len, unsigned long long* d_sum, hipStream_t s);
// Builds the chunk-major copy (fwd_ptr / fwd_term / fwd_w) from the postings and their
// weights; cnt is scratch of n_docs ints.
hipError_t sparse_forward(const SparseIndex& sp, int* cnt, hipStream_t s);
// Fills the dense head rows (whead, zeroed here) from the postings of the head terms
// head_terms[0 .. n_head) (device array, row h = term head_terms[h]).
hipError_t sparse_head_rows(const SparseIndex& sp, const int* head_terms, hipStream_t s);
size_t sparse_workspace_bytes(long long n_docs, int nq, int k);
hipError_t launch_sparse(const SparseIndex& sp, const int* qterm_indptr, const int* qterms, int nq, int k,
                         float* out_scores, long long* out_ids, void* ws, hipStream_t s);

// ---------------------------------------------------------------- fusion and upsert
// Dense-first hybrid: BM25 of the dense candidates cand [nq x n_cand] (dense order, -1 padded,
// 1 <= n_cand <= 128), reciprocal rank fusion with their dense order, top k.
// BM25 scores of every chunk [0, n_docs) for nq queries into dump [nq x ld], and the minimum
// and maximum over chunks [0, mm_rows) of each (query, range of kSparseRange chunks) into
// dump_mm [nq x ranges x 2] (+inf / -inf for a range with none of them).
// Weighted fusion inside the BM25 kernel when the corpus and the n scored chunks fit one
// range: the top k of w_d minmax(dense) + w_l minmax(BM25) over chunks [0, n).
hipError_t launch_sparse_weighted(const SparseIndex& sp, const int* qterm_indptr, const int* qterms, int nq, int k,
                                  const float* dense, long long ld, const float* dense_mm, int pd, long long n,
                                  double wd, double wl, float* out_scores, long long* out_ids, hipStream_t s);
// The hybrid's BM25 list and its reciprocal rank fusion with the dense list in one launch, when
// the corpus fits one range: the fused top k of each query.
hipError_t launch_sparse_rrf(const SparseIndex& sp, const int* qterm_indptr, const int* qterms, int nq, int k_sparse,
                             const long long* dense_ids, int k_dense, int rrf_k, int k, float* out_fused,
                             long long* out_ids, hipStream_t s);
hipError_t launch_sparse_dump(const SparseIndex& sp, const int* qterm_indptr, const int* qterms, int nq, float* dump,
                              long long ld, float* dump_mm, long long mm_rows, hipStream_t s);
hipError_t launch_dense_first(const SparseIndex& sp, const int* qterm_indptr, const int* qterms,
                              const long long* cand, int n_cand, long long nq, int rrf_k, int k, float* out_fused,
                              long long* out_ids, hipStream_t s);
hipError_t launch_rrf(const long long* dense_ids, int k_dense, const long long* sparse_ids, int k_sparse,
                      long long nq, int rrf_k, int k, float* out_fused, long long* out_ids, hipStream_t s);
// Mean pool over each chunk's first lengths[i] (clamped to [0, T]) tokens of hidden states
// [m x T x d] (bf16 or fp32), L2 normalisation, round to the slab dtype into rows
// [first_row, first_row + m).
hipError_t launch_pool_upsert(void* slab, int slab_dtype, int d, long long first_row, const void* hidden,
                              int hidden_dtype, const int* lengths, long long m, int T, hipStream_t s);
hipError_t launch_probe_read(const void* src, long long bytes, unsigned int* sink, int blocks, hipStream_t s);
hipError_t launch_upsert(void* slab, int slab_dtype, int d, long long first_row, const void* rows,
                         int rows_dtype, long long m, hipStream_t s);

}  // namespace oprag
