// Lexical retrieval: BM25 over an inverted-postings (CSR term -> (chunk, tf)) index that
// visits only the chunks containing a query term yet gives exact full-corpus BM25 scores
// (Section 4.4), with partial top-k selection instead of a full sort.
//
// Scoring reading (the paper does not fix the variant):
//   idf(t)  = ln(1 + (N - df + 0.5) / (df + 0.5)),  df = postings of t,  N = chunks;
//   score   = sum over query-term OCCURRENCES t of idf(t) tf (k1 + 1) / (tf + k1 (1 - b + b dl / avgdl)).
// Per-term factors idf(t)(k1 + 1) and per-posting weights tf / (tf + k1 (1 - b + b dl /
// avgdl)) are computed once in fp64 at attach time and stored as fp32, so a posting's
// contribution is one product; scores accumulate in fp32.
//
// One workgroup of 1,024 threads scores one query over a range of up to 32,768 chunks.  A
// query's distinct terms each contribute once, with m times their factor for m occurrences, in
// a fixed order: first the head terms (the most frequent ones, df >= N / 8, whose weights the
// attach keeps as dense per-chunk rows), then the others, each group in the query's
// first-occurrence order.  The head terms are summed from their rows in registers, each thread
// over its own 32 chunks (about nine in ten postings a batch touches belong to them, and walking
// them made every query read the same long lists again).  The remaining terms add their
// postings in the range to an fp32 accumulator in LDS (128 KiB), one term after another with a
// barrier in between, the next term's postings loading while the current one is added; a
// term's postings name distinct chunks, so there are no atomics and the result is
// deterministic.  The range's top-k then comes from a threshold (the k-th largest of the 256
// maxima of groups of four threads) and exact ranks of the few scores at or above it, with the
// keys held in registers; many scores above the threshold, or few positive ones, fall back to a
// 4 x 8-bit radix select and a wave-wide bitonic sort (score desc, chunk asc).
#include <algorithm>

#include "oprag_internal.h"
#include "rrf.h"
#include "select.h"

namespace oprag {
namespace {

using namespace dev;

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kBT = 1024;        // threads per scoring workgroup (sixteen waves on one CU)
constexpr int kNT = 256;         // threads per list-merge workgroup
constexpr int kTermBatch = kBT / 32;  // query terms whose posting bounds are found together

// Structural checks of the CSR, one thread per term, then one thread per posting (a posting
// finds its term by binary search over the offsets, so long lists are checked in parallel).
__global__ void validate_kernel(int vocab, long long n_docs, long long nnz, const long long* indptr,
                                const int* chunk, const int* tf, const int* doc_len, unsigned int* flag) {
  const long long tid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long stride = (long long)gridDim.x * blockDim.x;
  if (tid == 0 && (indptr[0] != 0 || indptr[vocab] != nnz)) atomicAdd(flag, 1u);
  for (long long t = tid; t < vocab; t += stride) {
    const long long lo = indptr[t], hi = indptr[t + 1];
    if (lo < 0 || hi < lo || hi > nnz) atomicAdd(flag, 1u);
  }
  for (long long p = tid; p < nnz; p += stride) {
    // term of posting p: the last t with indptr[t] <= p
    int lo = 0, hi = vocab;  // invariant: indptr[lo] <= p < indptr[hi] when the offsets are valid
    while (hi - lo > 1) {
      const int mid = lo + (hi - lo) / 2;
      if (indptr[mid] <= p)
        lo = mid;
      else
        hi = mid;
    }
    const int c = chunk[p];
    if (c < 0 || c >= n_docs || tf[p] < 1 || (p > indptr[lo] && chunk[p - 1] >= c)) atomicAdd(flag, 1u);
  }
  for (long long dd = tid; dd < n_docs; dd += stride)
    if (doc_len[dd] < 0) atomicAdd(flag, 1u);
}

__global__ void doclen_sum_kernel(const int* doc_len, long long n_docs, unsigned long long* sum) {
  __shared__ unsigned long long part[256];
  unsigned long long s = 0;
  for (long long i = threadIdx.x; i < n_docs; i += blockDim.x) s += (unsigned long long)doc_len[i];
  part[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long t = 0;
    for (int i = 0; i < 256; ++i) t += part[i];
    *sum = t;
  }
}

__global__ void prepare_kernel(int vocab, long long n_docs, long long nnz, const long long* indptr, const int* chunk,
                               const int* tf, const int* doc_len, double avgdl, double k1, double b, float* idfk,
                               float* wpost) {
  const long long tid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long stride = (long long)gridDim.x * blockDim.x;
  const double N = (double)n_docs;
  for (long long t = tid; t < vocab; t += stride) {
    const double df = (double)(indptr[t + 1] - indptr[t]);
    idfk[t] = (float)(log(1.0 + (N - df + 0.5) / (df + 0.5)) * (k1 + 1.0));
  }
  for (long long p = tid; p < nnz; p += stride) {
    const double f = (double)tf[p];
    wpost[p] = (float)(f / (f + k1 * (1.0 - b + b * (double)doc_len[chunk[p]] / avgdl)));
  }
}

// Block-wide exclusive prefix sum of one int per thread (kNT threads).
__device__ __forceinline__ int block_excl_scan(int v, int* wave_tot) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wave_tot[w] = x;
  __syncthreads();
  int before = 0;
  for (int i = 0; i < w; ++i) before += wave_tot[i];
  __syncthreads();
  return before + x - v;
}

struct SparseArgs {
  int vocab;
  long long n_docs;
  const long long* indptr;
  const int* chunk;
  const float* idfk;
  const float* wpost;
  const int* hidx;               // head row of each term, -1 for the others
  const float* whead;            // dense head rows [n_head x head_ld]
  long long head_ld;
  const int* qterm_indptr;
  const int* qterms;
  int nq;
  int k;
  int n_ranges;
  float* dump = nullptr;         // when set: every chunk's score to dump[q * dump_ld + chunk], no top-k
  long long dump_ld = 0;
  float* dump_mm = nullptr;      // with dump: (min, max) over chunks < mm_rows per (query, range)
  long long mm_rows = 0;
  // Weighted fusion in the kernel (one range): the top k of w_d minmax(dense) + w_l minmax(BM25)
  // over chunks [0, wn), the dense scores from wdense[q * wld + chunk] and their (min, max)
  // partials from wmm[(q * wpd + i) * 2 + {0, 1}], i < wpd.
  const float* wdense = nullptr;
  long long wld = 0;
  const float* wmm = nullptr;
  int wpd = 0;
  long long wn = 0;
  double wd = 0.0, wl = 0.0;
  // Hybrid fusion in the kernel (one range): the range's top k (the sparse list) stays in LDS
  // and is fused by reciprocal rank fusion with the dense list rrf_dense[q * rrf_kd ..] into
  // the top rrf_kout of rrf_fused / rrf_ids (rows of rrf_kout per query).
  const long long* rrf_dense = nullptr;
  int rrf_kd = 0;
  int rrf_k = 0;
  int rrf_kout = 0;
  float* rrf_fused = nullptr;
  long long* rrf_ids = nullptr;
  float* out_scores;            // final output when n_ranges == 1
  long long* out_ids;
  unsigned long long* partial;  // [nq x n_ranges x k] when n_ranges > 1
};

// Bounds [lo, hi) of the postings of one term whose chunks fall in [c0, c1), found by the 32
// threads of a group with a 32-ary search (three rounds for lists up to 32K postings).
// Every thread of the group returns the same bounds.
__device__ __forceinline__ void range_bounds32(const int* chunk, long long lo, long long hi, long long c0,
                                               long long c1, int sub, long long* out_lo, long long* out_hi) {
  long long a0 = lo, a1 = hi, b0 = lo, b1 = hi;  // first index >= c0 lies in [a0, a1]; >= c1 in [b0, b1]
  while (a1 - a0 > 0 || b1 - b0 > 0) {
    // probe 32 evenly spaced positions of each interval (step ceil(len / 32), so they reach
    // its end); the probes below the key form a prefix of the group
    const long long sa = (a1 - a0 + 31) / 32, sb = (b1 - b0 + 31) / 32;
    const long long pa = a0 + (long long)sub * sa, pb = b0 + (long long)sub * sb;
    const bool la = pa < a1 && chunk[pa] < c0;
    const bool lb = pb < b1 && chunk[pb] < c1;
    const unsigned long long ma = __ballot(la), mb = __ballot(lb);
    const int base = threadIdx.x & 32;  // this group's half of the wave
    const int ca = __popcll((ma >> base) & 0xffffffffull), cb = __popcll((mb >> base) & 0xffffffffull);
    if (a1 - a0 > 0) {
      if (ca == 0) a1 = a0;  // chunk[a0] >= c0
      else {
        const long long n0 = a0 + (long long)(ca - 1) * sa + 1;
        a1 = std::min(a1, a0 + (long long)ca * sa);
        a0 = n0;
      }
    }
    if (b1 - b0 > 0) {
      if (cb == 0) b1 = b0;
      else {
        const long long n0 = b0 + (long long)(cb - 1) * sb + 1;
        b1 = std::min(b1, b0 + (long long)cb * sb);
        b0 = n0;
      }
    }
  }
  *out_lo = a0;
  *out_hi = b0;
}

// Candidates the threshold selection ranks directly (their area also holds a query's head-term
// list while the scores are summed).  With the 128 KiB accumulator one workgroup fits a CU:
// a query of the 32K-chunk corpus takes one workgroup, one selection and no list merge.
constexpr int kCandCap = 992;

__global__ __launch_bounds__(kBT) void bm25_kernel(SparseArgs a) {
  __shared__ __attribute__((aligned(16))) float acc[kSparseRange];
  // One area, used in turn: the head-term list, the group maxima (threshold step), the
  // candidates (ranking), or the radix histogram and the winners (fallback path).
  __shared__ __attribute__((aligned(16))) u64 cand[kCandCap];
  unsigned int* hist = reinterpret_cast<unsigned int*>(cand);  // [256]
  u64* selbuf = cand + 128;                                    // [kMaxK]
  __shared__ int s_nc;
  __shared__ uint32_t s_tau;
  __shared__ int wave_tot[kBT / 64];
  __shared__ unsigned int s_prefix, s_need, s_take_all, s_ngt;
  __shared__ long long s_lo[kTermBatch], s_hi[kTermBatch];
  __shared__ float s_wt[kTermBatch];
  __shared__ long long s_sids[kMaxK];  // hybrid fusion: the sparse list by rank (-1 padded)
  static_assert(RrfScratch::kBytes <= kSparseRange * 4, "the fusion's scratch fits the accumulator");

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int q = blockIdx.x / a.n_ranges;
  const int range = blockIdx.x % a.n_ranges;
  const long long d0 = (long long)range * kSparseRange;
  const int len = (int)std::min<long long>(kSparseRange, a.n_docs - d0);
  // Thread tid owns the chunks 4 tid + kLayer g + e (g < 8 layers, e < 4) of the range: one
  // 16-byte column of each layer, so its head-row loads and key reads are whole 16-byte words.
  constexpr int kLayer = 4 * kBT;
  static_assert(kSparseRange == 8 * kLayer, "eight layers of four chunks per thread");
  auto own = [&](int j) { return 4 * tid + kLayer * (j >> 2) + (j & 3); };  // j < 32

  const int tb = a.qterm_indptr[q], te = a.qterm_indptr[q + 1];
  // With one range (a term's whole posting list is the range's) the parse pass also finds the
  // posting bounds of the tail terms among the first kTermBatch occurrences, so the first of
  // them is loading while the head rows are summed.
  const bool early = a.n_ranges == 1;
  // A term that occurs m times in the query takes part once, at its first occurrence, with
  // factor m * idf(t) (k1 + 1); unknown terms match nothing.
  // 1. head terms, from their dense rows.  The query's distinct head terms are listed in
  // first-occurrence order (in the candidate area, unused until the selection); then every
  // thread sums, term after term, the rows over its own chunks in registers.  A row holds 0
  // where the term is absent and fma(f, 0, s) = s, so these are exactly the fp32 operations of
  // walking the terms' postings, without searches, scattered LDS updates or barriers.
  int* hl_row = reinterpret_cast<int*>(cand);               // [kMaxHead]
  float* hl_wt = reinterpret_cast<float*>(cand) + kMaxHead;  // [kMaxHead]
  static_assert(2 * kMaxHead * 4 <= kCandCap * 8, "the head list fits the candidate area");
  int nh = 0;
  for (int j0 = tb; j0 < te; j0 += kBT) {
    const int j = j0 + tid;
    int row = -1;
    float wt = 0.f;
    long long tlo = 0, thi = 0;
    float twt = 0.f;
    if (j < te) {
      const int t = a.qterms[j];
      if (t >= 0 && t < a.vocab) {
        const int h = a.hidx[t];
        if (h >= 0 || (early && j < tb + kTermBatch)) {
          bool earlier = false;
          int mult = 0;
          for (int jj = tb; jj < te; ++jj)
            if (a.qterms[jj] == t) {
              if (jj < j) earlier = true;
              else ++mult;
            }
          if (!earlier) {
            if (h >= 0) {
              row = h;
              wt = a.idfk[t] * (float)mult;
            } else {
              tlo = a.indptr[t];
              thi = a.indptr[t + 1];
              twt = a.idfk[t] * (float)mult;
            }
          }
        }
      }
    }
    if (early && j0 == tb && tid < kTermBatch) {
      s_lo[tid] = tlo;
      s_hi[tid] = thi;
      s_wt[tid] = twt;
    }
    const int f = row >= 0 ? 1 : 0;
    const int pos = nh + block_excl_scan(f, wave_tot);
    if (f) {  // distinct head terms <= kMaxHead
      hl_row[pos] = row;
      hl_wt[pos] = wt;
    }
    if (tid == kBT - 1) s_nc = pos + f;  // the count so far, shared
    __syncthreads();
    nh = s_nc;
    __syncthreads();
  }

  // Tail postings, four per thread per step with every load issued before the first update.
  auto load_step = [&](long long p, long long hi, int (&c)[4], float (&wp)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const long long pu = p + (long long)u * kBT;
      c[u] = pu < hi ? a.chunk[pu] - (int)d0 : -1;
      wp[u] = pu < hi ? a.wpost[pu] : 0.f;
    }
  };
  auto apply_step = [&](float wt, const int (&c)[4], const float (&wp)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (c[u] >= 0) acc[c[u]] = __builtin_fmaf(wt, wp[u], acc[c[u]]);
  };
  auto next_term = [&](int g, int ng) {  // the first term from g on with postings (uniform)
    while (g < ng && !(s_lo[g] < s_hi[g])) ++g;
    return g;
  };
  int pc[4] = {-1, -1, -1, -1};  // the first step of the next tail term, in flight
  float pw[4] = {0.f, 0.f, 0.f, 0.f};
  int g_first = 0;
  if (early) {
    g_first = next_term(0, min(kTermBatch, te - tb));
    if (g_first < min(kTermBatch, te - tb)) load_step(s_lo[g_first] + tid, s_hi[g_first], pc, pw);
  }

  {
    f32x4 hs[8];
#pragma unroll
    for (int g = 0; g < 8; ++g) hs[g] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto load_row = [&](int i, f32x4 (&v)[8]) __attribute__((always_inline)) {
      const float* row = a.whead + (long long)hl_row[i] * a.head_ld + d0;
#pragma unroll
      for (int g = 0; g < 8; ++g) {
        const int c = 4 * tid + kLayer * g;  // d0 + c < n_docs: c .. c + 3 lie inside the padded row
        v[g] = c < len ? *reinterpret_cast<const f32x4*>(row + c) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    };
    auto add_row = [&](float wt, const f32x4 (&v)[8]) __attribute__((always_inline)) {
#pragma unroll
      for (int g = 0; g < 8; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) hs[g][e] = __builtin_fmaf(wt, v[g][e], hs[g][e]);
    };
    // the rows of two terms in flight at once
    int i = 0;
    for (; i + 1 < nh; i += 2) {
      f32x4 v0[8], v1[8];
      load_row(i, v0);
      load_row(i + 1, v1);
      add_row(hl_wt[i], v0);
      add_row(hl_wt[i + 1], v1);
    }
    if (i < nh) {
      f32x4 v0[8];
      load_row(i, v0);
      add_row(hl_wt[i], v0);
    }
    // every position of the accumulator is written, so chunks past len hold 0
#pragma unroll
    for (int g = 0; g < 8; ++g) *reinterpret_cast<f32x4*>(acc + 4 * tid + kLayer * g) = hs[g];
    __syncthreads();  // the accumulator is complete; the head list area is free again
  }

  // 2. the other (tail) terms, from their postings, one term after another (a term's postings
  // name distinct chunks: no atomics); the first step of the next term is loading while the
  // current one is added.
  for (int j0 = tb; j0 < te; j0 += kTermBatch) {
    const int ng = min(kTermBatch, te - j0);
    int g = g_first;
    if (!(early && j0 == tb)) {
      // posting bounds of up to kTermBatch terms at once, 32 threads per term
      __syncthreads();  // every thread is done with the previous batch's bounds
      const int gg = tid >> 5, sub = tid & 31;
      const int j = j0 + gg;
      static_assert(kTermBatch * 32 == kBT, "32 threads per term");
      long long lo = 0, hi = 0;
      float wt = 0.f;
      if (j < te) {  // uniform over the group's 32 threads
        const int t = a.qterms[j];
        if (t >= 0 && t < a.vocab) {
          int earlier = 0, mult = 0;
          for (int jj = tb + sub; jj < te; jj += 32)
            if (a.qterms[jj] == t) {
              if (jj < j) earlier = 1;
              else mult += 1;
            }
#pragma unroll
          for (int o = 16; o > 0; o >>= 1) {
            earlier |= __shfl_xor(earlier, o, 32);
            mult += __shfl_xor(mult, o, 32);
          }
          if (!earlier && a.hidx[t] < 0) {  // head terms were summed from their rows
            lo = a.indptr[t];
            hi = a.indptr[t + 1];
            wt = a.idfk[t] * (float)mult;
            if (a.n_ranges > 1) range_bounds32(a.chunk, lo, hi, d0, d0 + len, sub, &lo, &hi);
          }
        }
      }
      if (sub == 0) {
        s_lo[gg] = lo;
        s_hi[gg] = hi;
        s_wt[gg] = wt;
      }
      __syncthreads();
      g = next_term(0, ng);
      if (g < ng) load_step(s_lo[g] + tid, s_hi[g], pc, pw);
    }
    while (g < ng) {  // workgroup-uniform
      const long long lo = s_lo[g], hi = s_hi[g];
      const float wt = s_wt[g];
      const int gn = next_term(g + 1, ng);
      int nc[4] = {-1, -1, -1, -1};
      float nw[4] = {0.f, 0.f, 0.f, 0.f};
      if (gn < ng) load_step(s_lo[gn] + tid, s_hi[gn], nc, nw);
      apply_step(wt, pc, pw);
      for (long long p = lo + tid + 4 * kBT; p < hi; p += 4 * kBT) {
        int c[4];
        float wp[4];
        load_step(p, hi, c, wp);
        apply_step(wt, c, wp);
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        pc[u] = nc[u];
        pw[u] = nw[u];
      }
      g = gn;
    }
  }
  __syncthreads();
  if (a.dump != nullptr) {  // launch-uniform: the range's scores, no selection
    float* dst = a.dump + (long long)q * a.dump_ld + d0;
    const int mm_len = (int)std::max<long long>(0, std::min<long long>(len, a.mm_rows - d0));
    float mn = __builtin_inff(), mx = -__builtin_inff();
    for (int i = tid; i < len; i += kBT) {
      const float v = acc[i];
      dst[i] = v;
      if (i < mm_len) {
        mn = fminf(mn, v);
        mx = fmaxf(mx, v);
      }
    }
    if (a.dump_mm != nullptr) {  // launch-uniform
      for (int o = 32; o > 0; o >>= 1) {
        mn = fminf(mn, __shfl_xor(mn, o));
        mx = fmaxf(mx, __shfl_xor(mx, o));
      }
      float* red = reinterpret_cast<float*>(cand);  // [kBT / 64][2], the candidate area is unused here
      if (lane == 0) {
        red[2 * w] = mn;
        red[2 * w + 1] = mx;
      }
      __syncthreads();
      if (tid == 0) {
        for (int u = 1; u < kBT / 64; ++u) {
          mn = fminf(mn, red[2 * u]);
          mx = fmaxf(mx, red[2 * u + 1]);
        }
        float* o = a.dump_mm + ((long long)q * a.n_ranges + range) * 2;
        o[0] = mn;
        o[1] = mx;
      }
    }
    return;
  }

  // ---- exact top-k of the range's positive scores (positive fp32 bits order as uints)
  const uint32_t* keys = reinterpret_cast<const uint32_t*>(acc);
  uint32_t kv[32];  // this thread's keys, kv[j] = key of chunk own(j)
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    const uint4 x = reinterpret_cast<const uint4*>(acc)[tid + kBT * g];
    kv[4 * g] = x.x;
    kv[4 * g + 1] = x.y;
    kv[4 * g + 2] = x.z;
    kv[4 * g + 3] = x.w;
  }
  const bool weighted = a.wdense != nullptr;  // launch-uniform
  if (weighted) {
    // Weighted fusion: the lexical row is this range's scores (0 past the corpus) over chunks
    // [0, wn); both rows are min-max normalised over those chunks, the dense minimum and
    // maximum from the dump's partials.  Keys become score_key(fused), nonzero for every
    // chunk below wn (all are candidates), 0 past it; they replace the scores in LDS for the
    // selection below.
    float mnd = __builtin_inff(), mxd = -__builtin_inff(), mnl = __builtin_inff(), mxl = -__builtin_inff();
    for (int i = tid; i < a.wpd; i += kBT) {
      mnd = fminf(mnd, a.wmm[((long long)q * a.wpd + i) * 2]);
      mxd = fmaxf(mxd, a.wmm[((long long)q * a.wpd + i) * 2 + 1]);
    }
#pragma unroll
    for (int j = 0; j < 32; ++j)
      if (own(j) < a.wn) {
        mnl = fminf(mnl, __uint_as_float(kv[j]));
        mxl = fmaxf(mxl, __uint_as_float(kv[j]));
      }
    for (int o = 32; o > 0; o >>= 1) {
      mnd = fminf(mnd, __shfl_xor(mnd, o));
      mxd = fmaxf(mxd, __shfl_xor(mxd, o));
      mnl = fminf(mnl, __shfl_xor(mnl, o));
      mxl = fmaxf(mxl, __shfl_xor(mxl, o));
    }
    float* red = reinterpret_cast<float*>(cand);  // [4][kBT / 64]; the candidate area is free
    if (lane == 0) {
      red[w] = mnd;
      red[kBT / 64 + w] = mxd;
      red[2 * (kBT / 64) + w] = mnl;
      red[3 * (kBT / 64) + w] = mxl;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kBT / 64; ++u) {
      mnd = fminf(mnd, red[u]);
      mxd = fmaxf(mxd, red[kBT / 64 + u]);
      mnl = fminf(mnl, red[2 * (kBT / 64) + u]);
      mxl = fmaxf(mxl, red[3 * (kBT / 64) + u]);
    }
    const double sd = mxd > mnd ? a.wd / ((double)mxd - (double)mnd) : 0.0;
    const double sl = mxl > mnl ? a.wl / ((double)mxl - (double)mnl) : 0.0;
    const float* drow = a.wdense + (long long)q * a.wld;
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      const int c0 = 4 * tid + kLayer * g;  // 16-byte aligned: wld is a multiple of 4
      const f32x4 x = c0 < a.wn ? *reinterpret_cast<const f32x4*>(drow + c0) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = 4 * g + e;
        kv[j] = c0 + e < a.wn ? score_key(fused_value(sd, sl, mnd, mnl, x[e], __uint_as_float(kv[j]))) : 0u;
      }
      reinterpret_cast<uint4*>(acc)[tid + kBT * g] = make_uint4(kv[4 * g], kv[4 * g + 1], kv[4 * g + 2], kv[4 * g + 3]);
    }
    __syncthreads();  // the keys in LDS are complete; the reduction area is free again
  }
  // the score a key stands for
  auto key_value = [&](uint32_t k32) { return weighted ? key_score(k32) : __uint_as_float(k32); };
  // hybrid fusion: the ranks go to LDS (filled after the barriers of the selection below), then
  // every thread fuses them with the dense list, the accumulator serving as scratch
  const bool rrf = a.rrf_dense != nullptr;  // launch-uniform
  if (rrf)
    for (int i = tid; i < a.k; i += kBT) s_sids[i] = -1;
  auto rrf_tail = [&]() {
    __syncthreads();  // every rank is in LDS and every read of the keys is done
    rrf_query<kBT>(a.rrf_dense + (long long)q * a.rrf_kd, a.rrf_kd, s_sids, a.k, a.rrf_k, a.rrf_kout,
                   a.rrf_fused + (long long)q * a.rrf_kout, a.rrf_ids + (long long)q * a.rrf_kout,
                   RrfScratch(reinterpret_cast<unsigned char*>(acc)));
  };
  // chunks that hold keys: the range's, or in weighted mode every chunk below wn
  const int slen = weighted ? (int)a.wn : len;
  // Threshold: the 256 groups of four adjacent threads (128 chunks each) take their largest
  // key, and tau = the k-th largest of these maxima.  Every maximum is the key of its own
  // chunk, so at least k chunks score >= tau and the top k lie among them.  Each of a group's
  // threads counts the maxima above and equal to its group's in a quarter of the list.
  {
    uint32_t m = 0u;
#pragma unroll
    for (int j = 0; j < 32; ++j) m = max(m, kv[j]);
    m = max(m, (uint32_t)__shfl_xor((int)m, 1));
    m = max(m, (uint32_t)__shfl_xor((int)m, 2));
    const int grp = tid >> 2, sub = tid & 3;
    // four blocks of 64 maxima, 68 words apart, so the blocks the four threads read start in
    // different LDS banks
    uint32_t* gmax = reinterpret_cast<uint32_t*>(cand);
    if (sub == 0) gmax[(grp >> 6) * 68 + (grp & 63)] = m;
    if (tid == 0) {
      s_tau = 0u;
      s_nc = 0;
    }
    __syncthreads();
    int gt = 0, eq = 0;
    const uint4* blk = reinterpret_cast<const uint4*>(gmax + sub * 68);
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const uint4 x = blk[u];
      gt += (x.x > m ? 1 : 0) + (x.y > m ? 1 : 0) + (x.z > m ? 1 : 0) + (x.w > m ? 1 : 0);
      eq += (x.x == m ? 1 : 0) + (x.y == m ? 1 : 0) + (x.z == m ? 1 : 0) + (x.w == m ? 1 : 0);
    }
    gt += __shfl_xor(gt, 1);
    gt += __shfl_xor(gt, 2);
    eq += __shfl_xor(eq, 1);
    eq += __shfl_xor(eq, 2);
    if (sub == 0 && m != 0u && gt <= a.k - 1 && a.k - 1 < gt + eq) s_tau = m;  // the k-th largest maximum
    __syncthreads();
  }
  const uint32_t tau = s_tau;  // 0: fewer than k positive maxima
  auto emit = [&](int r, u64 key) __attribute__((always_inline)) {
    if (rrf) {
      s_sids[r] = (long long)comp_row(key);
    } else if (a.n_ranges == 1) {
      a.out_ids[(long long)q * a.k + r] = (long long)comp_row(key);
      a.out_scores[(long long)q * a.k + r] = key_value((uint32_t)(key >> 32));
    } else {
      a.partial[((long long)q * a.n_ranges + range) * a.k + r] = key;
    }
  };
  auto composite = [&](int i) __attribute__((always_inline)) {
    return ((u64)keys[i] << 32) | (uint32_t)(~(uint32_t)(d0 + i));
  };
  if (tau != 0u) {
    // G scores above tau and E equal to it.  When G + E fit the candidate area all of them
    // are ranked as unique composites (score, ~chunk), which orders equal scores by chunk.
    // Otherwise the G above tau are ranked and, when G < k, ranks G .. k - 1 go to the chunks
    // equal to tau in chunk order (many chunks can share a score exactly: equal term
    // frequencies and lengths).  G + E >= k always.
    uint32_t mgt = 0u, meq = 0u;
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      mgt |= (kv[j] > tau ? 1u : 0u) << j;
      meq |= (kv[j] == tau ? 1u : 0u) << j;
    }
    // both counts in one scan: G and E are at most 32,768, so the low field never carries
    const int packed = __popc(mgt) | (__popc(meq) << 16);
    const int before = block_excl_scan(packed, wave_tot);
    if (tid == kBT - 1) s_nc = before + packed;
    __syncthreads();
    const int G = s_nc & 0xffff, E = s_nc >> 16;
    const bool all = G + E <= kCandCap;  // workgroup-uniform
    if (G <= kCandCap) {
      int pos = all ? (before & 0xffff) + (before >> 16) : (before & 0xffff);
      for (uint32_t msk = all ? (mgt | meq) : mgt; msk != 0u; msk &= msk - 1u)
        cand[pos++] = composite(own(__builtin_ctz(msk)));
      __syncthreads();
      // rank = number of larger composites; L adjacent lanes share a candidate, each
      // comparing every L-th entry
      const int nc = all ? G + E : G;
      int lg = 0;
      while (lg < 4 && (nc << (lg + 1)) <= kBT) ++lg;
      const int L = 1 << lg, jc = tid >> lg, p = tid & (L - 1);
      int r = 0;
      u64 me = 0ull;
      if (jc < nc) {
        me = cand[jc];
        for (int o = p; o < nc; o += 8 * L) {
          u64 v[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) v[u] = cand[min(o + u * L, nc - 1)];
#pragma unroll
          for (int u = 0; u < 8; ++u) r += (o + u * L < nc && v[u] > me) ? 1 : 0;
        }
      }
      for (int s = 1; s < L; s <<= 1) r += __shfl_xor(r, s);
      if (jc < nc && p == 0 && r < a.k) emit(r, me);
      if (!all && G < a.k) {
        // ranks G .. k - 1: each thread marks the scores equal to tau in a contiguous block of
        // 32 chunks, read from a rotated start (lanes then hit different LDS banks), and emits
        // them in order after a scan of the counts
        const int b0 = min(slen, 32 * tid), nb = min(slen, b0 + 32) - b0;
        uint32_t mk = 0u;
        for (int i = 0; i < nb; ++i) {
          const int o = (i + tid) % nb;
          mk |= (keys[b0 + o] == tau ? 1u : 0u) << o;
        }
        int rr = G + block_excl_scan(__popc(mk), wave_tot);
        for (uint32_t m2 = mk; m2 != 0u && rr < a.k; m2 &= m2 - 1u) emit(rr++, composite(b0 + __builtin_ctz(m2)));
      }
      if (rrf) rrf_tail();
      return;
    }
    __syncthreads();  // the candidate area becomes the histogram
  }

  // ---- radix select of the k-th largest positive score (few positive maxima or many
  // candidates), over the keys held in registers
  if (tid == 0) {
    s_prefix = 0u;
    s_need = (unsigned)a.k;
    s_take_all = 0u;
  }
  __syncthreads();
  for (int pass = 0; pass < 4; ++pass) {
    if (s_take_all) break;  // block-uniform
    const int shift = 24 - 8 * pass;
    const uint32_t hmask = pass == 0 ? 0u : (0xffffffffu << (shift + 8));
    const uint32_t prefix = s_prefix;
    const unsigned int need = s_need;
    if (tid < 256) hist[tid] = 0u;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const uint32_t u = kv[j];
      if (u != 0u && (u & hmask) == prefix) atomicAdd(&hist[(u >> shift) & 255u], 1u);
    }
    __syncthreads();
    // threads 0 .. 255 (waves 0 .. 3): thread t holds bin 255 - t; its inclusive scan is the
    // number of keys in bins >= 255 - t
    int hd = 0, x = 0;
    if (tid < 256) {
      hd = (int)hist[255 - tid];
      x = hd;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
      }
      if (lane == 63) wave_tot[w] = x;
    }
    __syncthreads();
    if (tid < 256) {
      int before = 0;
      for (int i = 0; i < w; ++i) before += wave_tot[i];
      const int incl = before + x, above = incl - hd;
      if (tid == 255 && incl < (int)need) s_take_all = 1u;  // fewer than k positive scores (pass 0)
      if (above < (int)need && incl >= (int)need) {
        s_prefix = prefix | ((uint32_t)(255 - tid) << shift);
        s_need = need - (unsigned)above;
      }
    }
    __syncthreads();
  }
  const bool take_all = s_take_all != 0u;
  const uint32_t T = s_prefix;
  const unsigned int need_eq = take_all ? 0u : s_need;

  // ---- collect: every key > T, then the need_eq smallest chunk ids with key == T (contiguous
  // blocks of 32 chunks per thread, so a scan of the counts orders the equal keys by chunk)
  if (tid == 0) s_ngt = 0u;
  __syncthreads();
  const int b0 = min(slen, 32 * tid), b1 = min(slen, b0 + 32);
  int n_eq = 0;
  for (int i = b0; i < b1; ++i) {
    const uint32_t u = keys[i];
    if (u == 0u) continue;
    if (take_all ? true : u > T) {
      const unsigned int slot = atomicAdd(&s_ngt, 1u);
      selbuf[slot] = composite(i);
    } else if (u == T) {
      ++n_eq;
    }
  }
  const int before = block_excl_scan(n_eq, wave_tot);
  if (!take_all && n_eq && before < (int)need_eq) {
    const unsigned int ngt = (unsigned int)a.k - need_eq;
    int r = before;
    for (int i = b0; i < b1 && r < (int)need_eq; ++i) {
      if (keys[i] == T) {
        selbuf[ngt + r] = composite(i);
        ++r;
      }
    }
  }
  __syncthreads();
  const int nsel = take_all ? (int)s_ngt : a.k;

  // ---- sort the winners (<= 128) with wave 0 and write them out
  if (tid < 64) {
    u64 x0 = lane < nsel ? selbuf[lane] : 0ull;
    u64 x1 = lane + 64 < nsel ? selbuf[lane + 64] : 0ull;
    x0 = wave_sort64_desc(x0, lane);
    x1 = wave_sort64_desc(x1, lane);
    u64 q1 = 0ull;
    wave_merge128(x0, q1, x1, lane);
    // The stored key is the raw fp32 bit pattern of a positive score (score_key of the fused
    // value in weighted mode).
    if (rrf) {
      if (lane < a.k) s_sids[lane] = x0 ? (long long)comp_row(x0) : -1ll;
      if (lane + 64 < a.k) s_sids[lane + 64] = q1 ? (long long)comp_row(q1) : -1ll;
    } else if (a.n_ranges == 1) {
      const long long o = (long long)q * a.k;
      if (lane < a.k) {
        a.out_ids[o + lane] = x0 ? (long long)comp_row(x0) : -1ll;
        a.out_scores[o + lane] = x0 ? key_value((uint32_t)(x0 >> 32)) : -__builtin_inff();
      }
      if (lane + 64 < a.k) {
        a.out_ids[o + lane + 64] = q1 ? (long long)comp_row(q1) : -1ll;
        a.out_scores[o + lane + 64] = q1 ? key_value((uint32_t)(q1 >> 32)) : -__builtin_inff();
      }
    } else {
      unsigned long long* dst = a.partial + ((long long)q * a.n_ranges + range) * a.k;
      if (lane < a.k) dst[lane] = x0;
      if (lane + 64 < a.k) dst[lane + 64] = q1;
    }
  }
  if (rrf) rrf_tail();
}

// Merge of the per-range lists when they hold at most kMergeCap composites per query.  Each
// list is sorted (descending, empty 0 slots last) and the composites are unique, so the rank
// of entry p of list i in the merged order is p plus, for every other list, the number of its
// entries above it: a binary search in LDS.
constexpr int kMergeCap = 1024;
__global__ __launch_bounds__(kNT) void partial_rank_kernel(const unsigned long long* partial, int P, int kp, int nq,
                                                           int k, float* out_scores, long long* out_ids) {
  __shared__ u64 c[kMergeCap];
  __shared__ int s_nv;
  const int q = blockIdx.x, tid = threadIdx.x;
  if (q >= nq) return;
  const int n = P * kp;
  const unsigned long long* src = partial + (long long)q * n;
  if (tid == 0) s_nv = 0;
  __syncthreads();
  int nv = 0;
  for (int i = tid; i < n; i += kNT) {
    const u64 x = src[i];
    c[i] = x;
    nv += x != 0ull ? 1 : 0;
  }
  if (nv) atomicAdd(&s_nv, nv);
  __syncthreads();
  const int n_valid = s_nv;
  const long long o = (long long)q * k;
  for (int j = tid; j < n; j += kNT) {
    const u64 me = c[j];
    if (me == 0ull) continue;
    const int li = j / kp;
    int r = j - li * kp;
    for (int l = 0; l < P; ++l) {
      if (l == li) continue;
      int lo = 0, hi = kp;  // entries of list l above me form a prefix
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (c[l * kp + mid] > me) lo = mid + 1;
        else hi = mid;
      }
      r += lo;
    }
    if (r < k) {
      out_ids[o + r] = (long long)comp_row(me);
      out_scores[o + r] = __uint_as_float((uint32_t)(me >> 32));
    }
  }
  for (int r = n_valid + tid; r < k; r += kNT) {
    out_ids[o + r] = -1ll;
    out_scores[o + r] = -__builtin_inff();
  }
}

// Merge P partial lists of kp composites per query (raw positive-fp32 keys) into the top-k.
__global__ __launch_bounds__(64) void partial_merge_kernel(const unsigned long long* partial, int P, int kp, int nq,
                                                           int k, float* out_scores, long long* out_ids) {
  const int q = blockIdx.x, lane = threadIdx.x;
  if (q >= nq) return;
  u64 q0 = 0ull, q1 = 0ull;
  const long long n = (long long)P * kp;
  const unsigned long long* src = partial + (long long)q * n;
  for (long long base = 0; base < n; base += 64) {
    const u64 c = base + lane < n ? src[base + lane] : 0ull;
    wave_offer(q0, q1, c, queue_at(q0, q1, k - 1), lane);
  }
  const long long o = (long long)q * k;
  if (lane < k) {
    out_ids[o + lane] = q0 ? (long long)comp_row(q0) : -1ll;
    out_scores[o + lane] = q0 ? __uint_as_float((uint32_t)(q0 >> 32)) : -__builtin_inff();
  }
  if (lane + 64 < k) {
    out_ids[o + lane + 64] = q1 ? (long long)comp_row(q1) : -1ll;
    out_scores[o + lane + 64] = q1 ? __uint_as_float((uint32_t)(q1 >> 32)) : -__builtin_inff();
  }
}

// ------------------------------------------------------------------------------------
// Chunk-major copy of the postings (built once at attach) for the lexical scoring of given
// chunks: counts per chunk, exclusive prefix sums, then every posting placed in its chunk's
// list (positions by atomics, so a list is in no particular order; the CSR holds a
// (term, chunk) pair at most once, so a list holds each term at most once).
// ------------------------------------------------------------------------------------
__global__ void fwd_count_kernel(long long nnz, const int* __restrict__ chunk, int* cnt) {
  const long long stride = (long long)gridDim.x * blockDim.x;
  for (long long p = (long long)blockIdx.x * blockDim.x + threadIdx.x; p < nnz; p += stride) atomicAdd(&cnt[chunk[p]], 1);
}

// One workgroup: ptr[i] = sum of cnt[0 .. i), ptr[n] = total, in tiles of 1,024 x 4 counts.
__global__ __launch_bounds__(1024) void fwd_scan_kernel(long long n, const int* __restrict__ cnt, long long* ptr) {
  __shared__ long long part[1024];
  const int t = threadIdx.x;
  long long carry = 0;
  for (long long base = 0; base < n; base += 4096) {
    long long v[4], sum = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const long long i = base + (long long)t * 4 + u;
      v[u] = i < n ? cnt[i] : 0;
      sum += v[u];
    }
    part[t] = sum;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {  // inclusive scan of the 1,024 tile sums
      const long long x = t >= off ? part[t - off] : 0;
      __syncthreads();
      part[t] += x;
      __syncthreads();
    }
    long long excl = carry + part[t] - sum;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const long long i = base + (long long)t * 4 + u;
      if (i < n) ptr[i] = excl;
      excl += v[u];
    }
    carry += part[1023];
    __syncthreads();  // part is rewritten by the next tile
  }
  if (t == 0) ptr[n] = carry;
}

// Workgroups take terms in turn; a term's postings go to their chunks' lists.
__global__ void fwd_fill_kernel(int vocab, const long long* __restrict__ indptr, const int* __restrict__ chunk,
                                const float* __restrict__ wpost, const long long* __restrict__ ptr, int* fill,
                                int* fwd_term, float* fwd_w) {
  for (long long t = blockIdx.x; t < vocab; t += gridDim.x) {
    const long long p1 = indptr[t + 1];
    for (long long p = indptr[t] + threadIdx.x; p < p1; p += blockDim.x) {
      const int d = chunk[p];
      const long long pos = ptr[d] + atomicAdd(&fill[d], 1);
      fwd_term[pos] = (int)t;
      fwd_w[pos] = wpost[p];
    }
  }
}

// Dense head rows: row h holds the posting weight of term head_terms[h] for every chunk (the
// rows are zeroed first, so a chunk without the term reads 0).  One workgroup per head term.
__global__ void head_rows_kernel(const long long* indptr, const int* chunk, const float* wpost, const int* head_terms,
                                 long long ld, float* whead) {
  const int h = blockIdx.x;
  const int t = head_terms[h];
  float* row = whead + (long long)h * ld;
  for (long long p = indptr[t] + threadIdx.x; p < indptr[t + 1]; p += blockDim.x) row[chunk[p]] = wpost[p];
}

// ------------------------------------------------------------------------------------
// Dense-first hybrid (the serving schedule of Section 4.1, "Retrieval", measured in Section
// 5.5: lexical reranking of the dense top-n candidates only).  One workgroup of 1,024 threads
// per query: the eight threads (c, j) = (t / 8, t % 8) share the dense candidate of rank c + 1
// and read its chunk-major (term, weight) list together, entries j, j + 8, ..., comparing each
// entry with up to 32 query terms at a time held in LDS; a match stores the weight in the
// candidate's slot for that term.  Like bm25_kernel, a term that occurs m times in the query
// takes part once, at its first occurrence, with factor m * idf(t) (k1 + 1), and the
// candidate's score is fma(factor, weight, score) over the distinct terms, the head terms
// first and then the others, each in first-occurrence order: the same fp32 operations in the
// same order, so a candidate scores exactly what the full BM25 search gives its chunk.  Candidates at or past the sparse corpus's n_docs chunks
// hold no postings and score 0.  The candidates with a positive score are ranked by (score
// desc, id asc); reciprocal rank fusion of that order with the dense order, compared exactly
// as fractions (as rrf_kernel does), gives the top k.
// ------------------------------------------------------------------------------------
constexpr int kDfThreads = 1024;
constexpr int kRrfExactMax = 100000;  // below this rrf_k the fused quotients order exactly
constexpr int kDfCand = 128;
constexpr int kDfLanes = kDfThreads / kDfCand;
__global__ __launch_bounds__(kDfThreads) void dense_first_kernel(int vocab, long long n_docs,
                                                                 const int* __restrict__ hidx,
                                                                 const long long* __restrict__ fwd_ptr,
                                                                 const int* __restrict__ fwd_term,
                                                                 const float* __restrict__ idfk,
                                                                 const float* __restrict__ fwd_w,
                                                                 const int* qterm_indptr, const int* qterms,
                                                                 const long long* cand, int n_cand, int rrf_k, int k,
                                                                 float* out_fused, long long* out_ids) {
  constexpr int kTerms = 32;  // query term occurrences per pass
  static_assert(kTerms * 32 == kDfThreads, "32 threads find the multiplicity of each occurrence");
  __shared__ int qt_s[kTerms];    // the pass's distinct-term occurrences (-1: repeat or unknown)
  __shared__ float fw_s[kTerms];  // their factors m * idf(t) (k1 + 1)
  __shared__ int hd_s[kTerms];    // 1 for a head term
  __shared__ float wq[kDfCand][kTerms + 1];
  __shared__ float lex[kDfCand];
  __shared__ long long cid[kDfCand];
  __shared__ long long fnum[kDfCand];
  __shared__ long long fden[kDfCand];
  __shared__ double fval[kDfCand];
  __shared__ int s_nv;  // valid candidates (the dense list pads with -1 at its end)
  const long long q = blockIdx.x;
  const int t = threadIdx.x, c = t / kDfLanes, j = t % kDfLanes;
  const long long id = c < n_cand ? cand[q * n_cand + c] : -1;
  const bool has_terms = id >= 0 && id < n_docs;  // chunks past the sparse corpus have none
  const long long f0 = has_terms ? fwd_ptr[id] : 0, f1 = has_terms ? fwd_ptr[id + 1] : 0;
  float sc = 0.f;  // thread j == 0 of a candidate: its score
  const int tb = qterm_indptr[q], e_end = qterm_indptr[q + 1];
  // The head terms are summed first, then the others (the order of the full BM25 search).  A
  // query of at most kTerms occurrences walks the lists once and sums the two kinds from the
  // stored matches; a longer one walks them once per kind.
  const bool single = e_end - tb <= kTerms;
  // The first step of the candidate's list is loaded here, before the query-term setup and
  // its barrier, so its latency overlaps them; every later step (and every later walk of the
  // list) loads its own entries.
  constexpr int kStep = 16;
  int tm[kStep];
  float wt[kStep];
  auto load_step = [&](long long f) {
#pragma unroll
    for (int v = 0; v < kStep; ++v) {
      const long long g = f + v * kDfLanes;
      tm[v] = g < f1 ? fwd_term[g] : -1;
      wt[v] = g < f1 ? fwd_w[g] : 0.f;
    }
  };
  load_step(f0 + j);
  bool pre = true;  // tm / wt hold the first step of the list
  for (int pass = 0; pass < (single ? 1 : 2); ++pass)
  for (int e0 = tb; e0 < e_end; e0 += kTerms) {
    const int ne = min(kTerms, e_end - e0);
    {
      // occurrence u = t / 32 of the pass: is it its term's first, and how often does the
      // term occur from here on (32 threads scan the query's terms, as bm25_kernel does)
      const int u = t >> 5, sub = t & 31;
      int term = -1, earlier = 0, mult = 0;
      if (u < ne) {
        term = qterms[e0 + u];
        for (int jj = tb + sub; jj < e_end; jj += 32)
          if (qterms[jj] == term) {
            if (jj < e0 + u) earlier = 1;
            else mult += 1;
          }
      }
#pragma unroll
      for (int o = 16; o > 0; o >>= 1) {
        earlier |= __shfl_xor(earlier, o, 32);
        mult += __shfl_xor(mult, o, 32);
      }
      if (sub == 0) {
        // unknown terms match nothing; a term takes part in the pass of its kind
        const bool known = u < ne && !earlier && term >= 0 && term < vocab;
        const bool head = known && hidx[term] >= 0;
        const bool use = known && (single || head == (pass == 0));
        qt_s[u] = use ? term : -1;
        hd_s[u] = head ? 1 : 0;
        fw_s[u] = use ? idfk[term] * (float)mult : 0.f;
      }
    }
    for (int i = t; i < kDfCand * kTerms; i += kDfThreads) wq[i / kTerms][i % kTerms] = 0.f;
    __syncthreads();
    // sixteen entries per thread and step, all loads issued before any comparison; per query
    // term the weights of matching entries are summed (a list holds a term once, so the sum
    // is that weight or 0) and a match is stored
    for (long long f = f0 + j; f < f1; f += kStep * kDfLanes) {
      if (!pre) load_step(f);
      pre = false;
      for (int u = 0; u < ne; ++u) {
        const int tu = qt_s[u];
        if (tu < 0) continue;  // uniform: the term takes part at an earlier occurrence, or never
        float m = 0.f;
#pragma unroll
        for (int v = 0; v < kStep; ++v) m += tm[v] == tu ? wt[v] : 0.f;
        if (m != 0.f) wq[c][u] = m;
      }
    }
    __syncthreads();
    if (j == 0 && has_terms) {  // an unmatched term adds 0 exactly
      if (single) {
        for (int kind = 1; kind >= 0; --kind)  // head terms (kind 1) first
          for (int u = 0; u < ne; ++u)
            if (qt_s[u] >= 0 && hd_s[u] == kind) sc = __builtin_fmaf(fw_s[u], wq[c][u], sc);
      } else {  // this pass holds one kind only
        for (int u = 0; u < ne; ++u)
          if (qt_s[u] >= 0) sc = __builtin_fmaf(fw_s[u], wq[c][u], sc);
      }
    }
    __syncthreads();  // qt_s, fw_s and wq are rewritten by the next pass
  }
  if (t == 0) s_nv = 0;
  __syncthreads();
  if (j == 0) {
    lex[c] = id >= 0 ? sc : 0.f;
    cid[c] = id;
    if (id >= 0) atomicAdd(&s_nv, 1);
  }
  __syncthreads();
  // ranking: the eight threads of candidate c each compare it with 16 of the candidates
  // (u = 16 j .. 16 j + 15); the counts are summed across the eight adjacent lanes
  auto sum8 = [](int x) {
    x += __shfl_xor(x, 1);
    x += __shfl_xor(x, 2);
    x += __shfl_xor(x, 4);
    return x;
  };
  constexpr int kPer = kDfCand / kDfLanes;
  const float me = lex[c];
  int rs = 0;  // lexical rank among the candidates with a positive score (invalid ones score 0)
  if (id >= 0 && me > 0.f) {
#pragma unroll
    for (int v = 0; v < kPer; ++v) {
      const int u = j * kPer + v;
      const float o = lex[u];
      rs += (o > 0.f && (o > me || (o == me && cid[u] < id))) ? 1 : 0;
    }
  }
  rs = sum8(rs);
  if (j == 0 && id >= 0) {
    const long long a = (long long)rrf_k + c + 1;
    long long num = 1, den = a;
    if (me > 0.f) {
      const long long b = (long long)rrf_k + rs + 1;
      num = a + b;
      den = a * b;
    }
    fnum[c] = num;
    fden[c] = den;
    fval[c] = (double)num / (double)den;
  }
  __syncthreads();
  int r = 0;  // final rank: candidates that beat this one in (fused desc, id asc)
  long long n0 = 0, d0 = 1;
  if (id >= 0) {
    n0 = fnum[c];
    d0 = fden[c];
    const double v0 = fval[c];
#pragma unroll
    for (int v = 0; v < kPer; ++v) {
      const int u = j * kPer + v;
      const long long oi = cid[u];
      bool beats = false;
      if (oi >= 0) {
        if (rrf_k < kRrfExactMax) {
          // distinct fused values differ by at least (rrf_k + 129)^-4, more than the rounding
          // of the correctly rounded quotients, and equal values round alike
          const double fv = fval[u];
          beats = fv > v0 || (fv == v0 && oi < id);
        } else {
          const long long lhs = fnum[u] * d0, rhs = n0 * fden[u];
          beats = lhs > rhs || (lhs == rhs && oi < id);
        }
      }
      r += beats ? 1 : 0;
    }
  }
  r = sum8(r);
  if (j == 0 && id >= 0 && r < k) {
    out_ids[q * k + r] = id;
    out_fused[q * k + r] = (float)((double)n0 / (double)d0);
  }
  // slots past the valid candidates
  if (t < k) {
    const int nv = s_nv;
    if (t >= nv) {
      out_ids[q * k + t] = -1;
      out_fused[q * k + t] = -__builtin_inff();
    }
  }
}

}  // namespace

hipError_t sparse_validate(int vocab, long long n_docs, long long nnz, const long long* indptr, const int* chunk,
                           const int* tf, const int* doc_len, unsigned int* d_flag, hipStream_t s) {
  hipError_t e = hipMemsetAsync(d_flag, 0, sizeof(unsigned int), s);
  if (e != hipSuccess) return e;
  const long long work = std::max<long long>(std::max<long long>(vocab, n_docs), nnz);
  const int blocks = (int)std::min<long long>(1024, (work + 255) / 256);
  hipLaunchKernelGGL(validate_kernel, dim3(std::max(1, blocks)), dim3(256), 0, s, vocab, n_docs, nnz, indptr, chunk,
                     tf, doc_len, d_flag);
  return hipGetLastError();
}

hipError_t sparse_prepare(SparseIndex& sp, const int* doc_len, unsigned long long* dsum, hipStream_t s) {
  hipLaunchKernelGGL(doclen_sum_kernel, dim3(1), dim3(256), 0, s, doc_len, sp.n_docs, dsum);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  unsigned long long total = 0;
  e = hipMemcpyAsync(&total, dsum, sizeof(total), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return e;
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return e;
  sp.avgdl = (double)total / (double)sp.n_docs;
  const long long work = std::max<long long>(sp.vocab, sp.nnz);
  const int blocks = (int)std::min<long long>(4096, (work + 255) / 256);
  hipLaunchKernelGGL(prepare_kernel, dim3(std::max(1, blocks)), dim3(256), 0, s, sp.vocab, sp.n_docs, sp.nnz,
                     sp.term_indptr, sp.post_chunk, sp.post_tf, doc_len, sp.avgdl, (double)sp.k1, (double)sp.b, sp.idfk,
                     sp.wpost);
  return hipGetLastError();
}

hipError_t sparse_forward(const SparseIndex& sp, int* cnt, hipStream_t s) {
  hipError_t e = hipMemsetAsync(cnt, 0, (size_t)sp.n_docs * sizeof(int), s);
  if (e != hipSuccess) return e;
  const int blocks = (int)std::min<long long>(4096, std::max<long long>(1, (sp.nnz + 255) / 256));
  hipLaunchKernelGGL(fwd_count_kernel, dim3(blocks), dim3(256), 0, s, sp.nnz, sp.post_chunk, cnt);
  hipLaunchKernelGGL(fwd_scan_kernel, dim3(1), dim3(1024), 0, s, sp.n_docs, cnt, sp.fwd_ptr);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipMemsetAsync(cnt, 0, (size_t)sp.n_docs * sizeof(int), s);
  if (e != hipSuccess) return e;
  const int tblocks = (int)std::min<long long>(65536, std::max(1, sp.vocab));
  hipLaunchKernelGGL(fwd_fill_kernel, dim3(tblocks), dim3(256), 0, s, sp.vocab, sp.term_indptr, sp.post_chunk,
                     sp.wpost, sp.fwd_ptr, cnt, sp.fwd_term, sp.fwd_w);
  return hipGetLastError();
}

hipError_t sparse_head_rows(const SparseIndex& sp, const int* head_terms, hipStream_t s) {
  hipError_t e = hipMemsetAsync(sp.whead, 0, (size_t)sp.n_head * (size_t)sp.head_ld * sizeof(float), s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(head_rows_kernel, dim3((unsigned)sp.n_head), dim3(256), 0, s, sp.term_indptr, sp.post_chunk,
                     sp.wpost, head_terms, sp.head_ld, sp.whead);
  return hipGetLastError();
}

hipError_t launch_sparse_dump(const SparseIndex& sp, const int* qterm_indptr, const int* qterms, int nq, float* dump,
                              long long ld, float* dump_mm, long long mm_rows, hipStream_t s) {
  SparseArgs a;
  a.vocab = sp.vocab;
  a.n_docs = sp.n_docs;
  a.indptr = sp.term_indptr;
  a.chunk = sp.post_chunk;
  a.idfk = sp.idfk;
  a.wpost = sp.wpost;
  a.hidx = sp.hidx;
  a.whead = sp.whead;
  a.head_ld = sp.head_ld;
  a.qterm_indptr = qterm_indptr;
  a.qterms = qterms;
  a.nq = nq;
  a.k = 1;
  a.n_ranges = (int)((sp.n_docs + kSparseRange - 1) / kSparseRange);
  a.dump = dump;
  a.dump_ld = ld;
  a.dump_mm = dump_mm;
  a.mm_rows = mm_rows;
  a.out_scores = nullptr;
  a.out_ids = nullptr;
  a.partial = nullptr;
  hipLaunchKernelGGL(bm25_kernel, dim3((unsigned)(nq * a.n_ranges)), dim3(kBT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sparse_weighted(const SparseIndex& sp, const int* qterm_indptr, const int* qterms, int nq, int k,
                                  const float* dense, long long ld, const float* dense_mm, int pd, long long n,
                                  double wd, double wl, float* out_scores, long long* out_ids, hipStream_t s) {
  if (sp.n_docs > kSparseRange || n > kSparseRange || ld % 4) return hipErrorInvalidValue;
  SparseArgs a;
  a.vocab = sp.vocab;
  a.n_docs = sp.n_docs;
  a.indptr = sp.term_indptr;
  a.chunk = sp.post_chunk;
  a.idfk = sp.idfk;
  a.wpost = sp.wpost;
  a.hidx = sp.hidx;
  a.whead = sp.whead;
  a.head_ld = sp.head_ld;
  a.qterm_indptr = qterm_indptr;
  a.qterms = qterms;
  a.nq = nq;
  a.k = k;
  a.n_ranges = 1;
  a.wdense = dense;
  a.wld = ld;
  a.wmm = dense_mm;
  a.wpd = pd;
  a.wn = n;
  a.wd = wd;
  a.wl = wl;
  a.out_scores = out_scores;
  a.out_ids = out_ids;
  a.partial = nullptr;
  hipLaunchKernelGGL(bm25_kernel, dim3((unsigned)nq), dim3(kBT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sparse_rrf(const SparseIndex& sp, const int* qterm_indptr, const int* qterms, int nq, int k_sparse,
                             const long long* dense_ids, int k_dense, int rrf_k, int k, float* out_fused,
                             long long* out_ids, hipStream_t s) {
  if (sp.n_docs > kSparseRange) return hipErrorInvalidValue;
  SparseArgs a;
  a.vocab = sp.vocab;
  a.n_docs = sp.n_docs;
  a.indptr = sp.term_indptr;
  a.chunk = sp.post_chunk;
  a.idfk = sp.idfk;
  a.wpost = sp.wpost;
  a.hidx = sp.hidx;
  a.whead = sp.whead;
  a.head_ld = sp.head_ld;
  a.qterm_indptr = qterm_indptr;
  a.qterms = qterms;
  a.nq = nq;
  a.k = k_sparse;
  a.n_ranges = 1;
  a.rrf_dense = dense_ids;
  a.rrf_kd = k_dense;
  a.rrf_k = rrf_k;
  a.rrf_kout = k;
  a.rrf_fused = out_fused;
  a.rrf_ids = out_ids;
  a.out_scores = nullptr;
  a.out_ids = nullptr;
  a.partial = nullptr;
  hipLaunchKernelGGL(bm25_kernel, dim3((unsigned)nq), dim3(kBT), 0, s, a);
  return hipGetLastError();
}

size_t sparse_workspace_bytes(long long n_docs, int nq, int k) {
  const long long n_ranges = (n_docs + kSparseRange - 1) / kSparseRange;
  if (n_ranges <= 1) return 0;
  return (size_t)nq * (size_t)n_ranges * (size_t)k * sizeof(unsigned long long);
}

hipError_t launch_sparse(const SparseIndex& sp, const int* qterm_indptr, const int* qterms, int nq, int k,
                         float* out_scores, long long* out_ids, void* ws, hipStream_t s) {
  SparseArgs a;
  a.vocab = sp.vocab;
  a.n_docs = sp.n_docs;
  a.indptr = sp.term_indptr;
  a.chunk = sp.post_chunk;
  a.idfk = sp.idfk;
  a.wpost = sp.wpost;
  a.hidx = sp.hidx;
  a.whead = sp.whead;
  a.head_ld = sp.head_ld;
  a.qterm_indptr = qterm_indptr;
  a.qterms = qterms;
  a.nq = nq;
  a.k = k;
  a.n_ranges = (int)((sp.n_docs + kSparseRange - 1) / kSparseRange);
  a.out_scores = out_scores;
  a.out_ids = out_ids;
  a.partial = static_cast<unsigned long long*>(ws);
  hipLaunchKernelGGL(bm25_kernel, dim3((unsigned)(nq * a.n_ranges)), dim3(kBT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_ranges == 1) return e;
  if ((long long)a.n_ranges * k <= kMergeCap)
    hipLaunchKernelGGL(partial_rank_kernel, dim3((unsigned)nq), dim3(kNT), 0, s, a.partial, a.n_ranges, k, nq, k,
                       out_scores, out_ids);
  else
    hipLaunchKernelGGL(partial_merge_kernel, dim3((unsigned)nq), dim3(64), 0, s, a.partial, a.n_ranges, k, nq, k,
                       out_scores, out_ids);
  return hipGetLastError();
}

hipError_t launch_dense_first(const SparseIndex& sp, const int* qterm_indptr, const int* qterms,
                              const long long* cand, int n_cand, long long nq, int rrf_k, int k, float* out_fused,
                              long long* out_ids, hipStream_t s) {
  if (n_cand < 1 || n_cand > kDfCand) return hipErrorInvalidValue;
  hipLaunchKernelGGL(dense_first_kernel, dim3((unsigned)nq), dim3(kDfThreads), 0, s, sp.vocab, sp.n_docs, sp.hidx,
                     sp.fwd_ptr, sp.fwd_term, sp.idfk, sp.fwd_w, qterm_indptr, qterms, cand, n_cand, rrf_k, k,
                     out_fused, out_ids);
  return hipGetLastError();
}

}  // namespace oprag
