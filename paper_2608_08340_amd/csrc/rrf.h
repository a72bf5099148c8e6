// Reciprocal rank fusion of one query's dense and sparse top lists (the hybrid's fusion step),
// shared by rrf_kernel and by the BM25 kernel's hybrid mode.
//
// fused(d) = sum over the lists L holding d of 1 / (k_rrf + rank_L(d)), 1-based ranks over a
// list's valid prefix (Cormack, Clarke and Buettcher, SIGIR 2009).  Fused values compare
// exactly as fractions num / den in 64-bit integers (den = the product of at most two
// (k_rrf + rank) factors), so exact ties such as 1/63 = 2/126 stay ties, broken by ascending id.
//
// Thread t < kd inserts dense entry t (rank t + 1) and thread kd + j sparse entry j (rank
// j + 1) into an LDS hash table keyed by id (open addressing, 64-bit compare-and-swap on the
// key), so an id present in both lists ends in one slot holding both ranks; the expected probe
// count is about one.  An occupied slot whose fused value reaches 1 / (rrf_k + k) is a
// candidate; its rank is the number of candidates that beat it in the exact rational order
// (fused desc, id asc), counted with LDS reads issued ahead of use.
#pragma once

#include "oprag_internal.h"

namespace oprag {
namespace dev {

constexpr int kRrfSlots = 512;       // power of two, at least twice the 256 possible ids
constexpr int kRrfMaxCand = 2 * kMaxK;
constexpr int kRrfFastMax = 100000;  // below this rrf_k the fused quotients order exactly

// LDS the fusion of one query uses (any 16-byte aligned area of at least kBytes).
struct RrfScratch {
  static constexpr int kBytes = kRrfSlots * 8 + 2 * kRrfSlots * 4 + kRrfMaxCand * 32 + 16;
  unsigned long long* key;  // [kRrfSlots] id, or ~0 when empty
  int* rank_d;              // [kRrfSlots]
  int* rank_s;              // [kRrfSlots]
  long long* cid;           // [kRrfMaxCand]
  long long* cnum;
  long long* cden;
  double* cval;
  int* nc;
  __device__ explicit RrfScratch(unsigned char* area)
      : key(reinterpret_cast<unsigned long long*>(area)),
        rank_d(reinterpret_cast<int*>(area + kRrfSlots * 8)),
        rank_s(reinterpret_cast<int*>(area + kRrfSlots * 12)),
        cid(reinterpret_cast<long long*>(area + kRrfSlots * 16)),
        cnum(reinterpret_cast<long long*>(area + kRrfSlots * 16 + kRrfMaxCand * 8)),
        cden(reinterpret_cast<long long*>(area + kRrfSlots * 16 + kRrfMaxCand * 16)),
        cval(reinterpret_cast<double*>(area + kRrfSlots * 16 + kRrfMaxCand * 24)),
        nc(reinterpret_cast<int*>(area + kRrfSlots * 16 + kRrfMaxCand * 32)) {}
};

// The fused top k of one query (its lists dense[0 .. kd) and sparse[0 .. ks), -1 padded; kd,
// ks <= kMaxK; either pointer may address global memory or LDS) to out_fused[0 .. k) and
// out_ids[0 .. k).  Called by every thread of an NT-thread workgroup (NT >= 256).
template <int NT>
__device__ void rrf_query(const long long* dense, int kd, const long long* sparse, int ks, int rrf_k, int k,
                          float* out_fused, long long* out_ids, const RrfScratch& sc) {
  static_assert(NT >= kRrfMaxCand, "a thread per list entry");
  constexpr unsigned long long kEmpty = ~0ull;
  unsigned long long* key = sc.key;
  int* rank_d = sc.rank_d;
  int* rank_s = sc.rank_s;
  long long* cid = sc.cid;
  long long* cnum = sc.cnum;
  long long* cden = sc.cden;
  double* cval = sc.cval;
  const int t = threadIdx.x;
  for (int h = t; h < kRrfSlots; h += NT) {
    key[h] = kEmpty;
    rank_d[h] = 0;
    rank_s[h] = 0;
  }
  if (t == 0) *sc.nc = 0;
  long long id = -1;
  int rank = 0;
  bool is_dense = false;
  if (t < kd) {
    id = dense[t];
    rank = t + 1;
    is_dense = true;
  } else if (t - kd < ks) {
    id = sparse[t - kd];
    rank = t - kd + 1;
  }
  __syncthreads();
  if (id >= 0) {
    unsigned h = ((unsigned)id * 2654435761u) >> 23;  // top 9 bits
    for (;;) {  // at most 256 ids in 512 slots: a free or matching slot is always found
      const unsigned long long old = atomicCAS(&key[h], kEmpty, (unsigned long long)id);
      if (old == kEmpty || old == (unsigned long long)id) break;
      h = (h + 1) & (kRrfSlots - 1);
    }
    if (is_dense)
      rank_d[h] = rank;
    else
      rank_s[h] = rank;
  }
  __syncthreads();
  // compaction; fused = 1/(rrf_k + a) + 1/(rrf_k + b) = num / den exactly
  for (int h = t; h < kRrfSlots; h += NT) {
    if (key[h] != kEmpty) {
      const long long a = rank_d[h] ? (long long)rrf_k + rank_d[h] : 0, b = rank_s[h] ? (long long)rrf_k + rank_s[h] : 0;
      long long num, den;
      if (a && b) {
        num = a + b;
        den = a * b;
      } else {
        num = 1;
        den = a ? a : b;
      }
      // The entries of rank <= k of either list all fuse to >= 1 / (rrf_k + k), and there
      // are at least min(k, candidates) of them, so a candidate below that never ranks < k.
      if (num * ((long long)rrf_k + k) >= den) {
        const int slot = atomicAdd(sc.nc, 1);
        cid[slot] = (long long)key[h];
        cnum[slot] = num;
        cden[slot] = den;
        cval[slot] = (double)num / (double)den;
      }
    }
  }
  __syncthreads();
  const int nc = *sc.nc;
  if (t < nc) {
    // Rank = candidates that beat this one.
    const long long n0 = cnum[t], d0 = cden[t], id0 = cid[t];
    const double v0 = cval[t];
    int r = 0;
    if (rrf_k < kRrfFastMax) {
      // Distinct fused values differ by at least 1 / (den1 den2) >= (rrf_k + 128)^-4, more
      // than twice the rounding error of the correctly rounded quotients (about
      // 2 / (rrf_k + 1) * 2^-53) while rrf_k stays below ~1.6e5; equal values round alike.
      // So the quotients order the candidates exactly, and their bit patterns (positive
      // doubles) order like unsigned integers.  Eight candidates per step, read before use.
      const unsigned long long b0 = (unsigned long long)__double_as_longlong(v0);
      for (int o = 0; o < nc; o += 8) {
        unsigned long long vb[8];
        long long ii[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int c = min(o + u, nc - 1);
          vb[u] = (unsigned long long)__double_as_longlong(cval[c]);
          ii[u] = cid[c];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) r += (o + u < nc && (vb[u] > b0 || (vb[u] == b0 && ii[u] < id0))) ? 1 : 0;
      }
    } else {
      // Large rrf_k: the quotients order pairs that differ by more than a few ulps; closer
      // pairs are compared exactly as int64 cross products.
      const double hi = v0 * (1.0 + 1e-14), lo = v0 * (1.0 - 1e-14);
      for (int o = 0; o < nc; o += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (o + u < nc) {
            const double v = cval[o + u];
            bool beats = v > hi;
            if (!beats && v >= lo) {
              const long long lhs = cnum[o + u] * d0, rhs = n0 * cden[o + u];
              beats = lhs > rhs || (lhs == rhs && cid[o + u] < id0);
            }
            r += beats ? 1 : 0;
          }
        }
      }
    }
    if (r < k) {
      out_ids[r] = id0;
      out_fused[r] = (float)((double)n0 / (double)d0);
    }
  }
  for (int r = nc + t; r < k; r += NT) {
    out_ids[r] = -1;
    out_fused[r] = -__builtin_inff();
  }
}

}  // namespace dev
}  // namespace oprag
