// Dense exact top-k: R_k = Op_retrieve(q, I) (Section 3.2, "Retrieval"): inner-product
// scores of every query against every indexed unit vector, by matrix products over the
// embedding matrix, then partial top-k selection (Section 4.4).
//
// The grid is (row chunk) x (query block).  Each workgroup streams its chunk of rows tile by
// tile, scores a tile against its query block with MFMA (bf16 / fp16 storage, fp32
// accumulation) or VALU FMA (fp32 storage), keeps a per-query top-k across its tiles, and
// writes that local top-k to its own slot of a partial-list buffer (no atomics, no
// cross-workgroup traffic).  A second, small kernel merges the chunk lists of each query;
// with a single chunk the first kernel writes the final list itself.  The score matrix
// never leaves the chip.
//
// Data movement for bf16 / fp16: each wave owns MW 16-row subtiles of a tile and loads their
// rows with 16-byte buffer loads straight into VGPRs, already in the MFMA A-operand layout
// (lane l: row l % 16, eight dimensions 8 (l / 16) of a 32-dimension k-step); a register ring
// of RS k-steps keeps RS - 1 of them in flight.  The query block is shared by the waves: each
// 128-dimension super-step of it is loaded one super-step ahead into VGPRs and written to one
// of two LDS slots (16-byte pieces swizzled by row so writes and fragment reads use all
// banks), from which every wave reads its B operands one k-step ahead of the MFMAs.
//
// Selection (k <= 16) runs after each tile on the accumulators.  A chunk's first tile, and
// any tile the faster test declines, takes the group path: the k-th largest of the lanes'
// group maxima (with the running list) bounds the k-th best score from below, only the
// scores reaching it go to LDS, and each query's owner thread inserts them into its running
// (score desc, id asc) list of 64-bit composites.  Later tiles compare each lane's group
// maximum with the running k-th score and hand over the rare hits.  Heavy ties fall back to
// passes over an LDS score tile: the top-KS values of each slice (a v_med3 insertion
// network), then the rows above the exact k-th value and the smallest-id rows equal to it.
// Filtered mode (bf16 / fp16, 16 < k <= 128): threshold levels over growing row prefixes
// collect candidate keys per query (a kernel instance with branch-free stores for levels with
// many hits per tile, SEL 4, and one with per-hit stores for the others, SEL 2) and
// select_topk_kernel ranks them.  fp32 with k > 16: one
// wave per query keeps a 128-entry sorted queue and merges batches of 64 candidates above
// its k-th entry with a bitonic network.
#include <algorithm>

#include <hip/hip_ext.h>

#include "oprag_internal.h"
#include "select.h"

namespace oprag {

// The top-5 list kernels for batches up to 16 and above 128 are compiled a second time, in
// dense_ilp.hip, under the machine scheduler that favours instruction-level parallelism, and
// the kernel table points at those instances: their calls take 2 % less time with it (batches
// 1, 16 and 256), while the 64-query top-5 kernels and the filtered ones take longer (1 to 7 %)
// and the 65-128-query one the same, and keep the default.  X(DT, NW, MW, RS, G, KS, SEL, WV,
// QR) for each.
#define OPRAG_ILP_KERNELS(X, DT)                                                                   \
  X(DT, 1, 1, 16, 1, 5, 0, 4, 8) X(DT, 1, 1, 16, 1, 5, 0, 4, 0) X(DT, 1, 1, 4, 1, 5, 0, 4, 0)     \
  X(DT, 8, 4, 4, 2, 5, 0, 4, 0)
template <int DT, int NW, int MW, int RS, int G, int KS, int SEL, int WV, int QR>
__global__ __launch_bounds__(WV * 64) void dense_mfma_kernel_ilp(DenseArgs a);

namespace {

using namespace dev;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int DT>
struct Mfma;
template <>
struct Mfma<kDtypeBF16> {
  typedef bf16x8 V;
  typedef __bf16 T;
  static __device__ __forceinline__ f32x4 run(V a, V b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mfma<kDtypeF16> {
  typedef f16x8 V;
  typedef _Float16 T;
  static __device__ __forceinline__ f32x4 run(V a, V b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
};

// Raw buffer resource over [base, base + bytes): 16-byte loads at offsets past the end
// return zeros instead of touching memory (gfx9 descriptor word 3: 32-bit data format).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, long long bytes) {
  const int n = (int)(unsigned)(bytes < 0 ? 0 : (bytes > 0xffffffffll ? 0xffffffffll : bytes));
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, int voffset) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voffset, 0, 0);
}

// Workgroup barrier that leaves in-flight ring loads in flight (a full __syncthreads()
// fence would drain them): this wave's LDS traffic is complete first.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Barrier after which every wave's global and LDS traffic is complete.
__device__ __forceinline__ void full_barrier() {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr float kNegInf = -__builtin_inff();

// Logical workgroup index with consecutive indices kept on one XCD (the hardware deals
// workgroups round-robin over the 8 XCDs), so the query blocks of one row chunk share an L2.
__device__ __forceinline__ long long logical_block() {
  const long long g = blockIdx.x, G = gridDim.x;
  return (G % 8 == 0) ? (g % 8) * (G / 8) + g / 8 : g;
}

// Top-KS values, sorted descending: new[i] = med3(v[i-1], v[i], x) = max(v[i], min(v[i-1], x)).
template <int KS>
struct ValTop {
  float v[KS];
  __device__ __forceinline__ void clear() {
#pragma unroll
    for (int i = 0; i < KS; ++i) v[i] = kNegInf;
  }
  __device__ __forceinline__ void insert(float x) {
#pragma unroll
    for (int i = KS - 1; i > 0; --i) v[i] = __builtin_amdgcn_fmed3f(v[i - 1], v[i], x);
    v[0] = __builtin_fmaxf(v[0], x);
  }
  __device__ __forceinline__ float at(int k) const {  // v[k - 1], k runtime
    float r = kNegInf;
#pragma unroll
    for (int i = 0; i < KS; ++i)
      if (i == k - 1) r = v[i];
    return r;
  }
};

// ------------------------------------------------------------------------------------
// Score tile in LDS, query-major: S[q * SR + rloc], rloc = position of a row in the pass.
// A pass holds the rows of one group of subtiles; rloc -> row id is increasing.
// ------------------------------------------------------------------------------------
struct PassRows {
  long long tile0;  // first row of the tile
  int blk;          // rows per block of the pass (a power of two)
  int blk_stride;   // row distance between consecutive blocks
  int off;          // row offset of the pass inside each block
  int nvalid;       // rloc < nvalid are rows below the row limit (a prefix: the map increases)
  __device__ __forceinline__ long long row(int rloc) const {
    return tile0 + (long long)(rloc / blk) * blk_stride + off + (rloc % blk);
  }
};

// k <= KS <= 16.  Scratch in LDS: candidates [BN][CAP] u64 | values [TPQ][BN][KS] f32 |
// per-thread counts [TPQ][BN] | tau [BN] | need [BN] | count [BN] | flag.
template <int BN, int KS, int NT>
struct SelSmall {
  static constexpr int TPQ = NT / BN;  // threads per query: t = q + BN * sub
  static constexpr int CAP = 2 * KS > 16 ? 2 * KS : 16;  // candidate slots per query and pass
  static constexpr int NL = KS <= 8 ? 4 : 2;             // independent value lists per thread
  static constexpr int kVals = TPQ > 1 ? TPQ * BN * KS * 4 : 0;
  static constexpr int kBytes = BN * CAP * 8 + kVals + TPQ * BN * 4 + BN * 12 + 16;
  RegTopK<KS> run;  // running list of the query (owner thread, sub == 0)

  __device__ __forceinline__ void init() { run.clear(); }

  // scratch regions shared with the register epilogue of the MFMA kernel
  static __device__ __forceinline__ u64* cand_of(unsigned char* sc) { return reinterpret_cast<u64*>(sc); }
  static __device__ __forceinline__ float* tau_of(unsigned char* sc) {
    return reinterpret_cast<float*>(sc + BN * CAP * 8 + kVals + TPQ * BN * 4);
  }
  static __device__ __forceinline__ int* cnt_of(unsigned char* sc) {
    return reinterpret_cast<int*>(sc + BN * CAP * 8 + kVals + TPQ * BN * 4 + BN * 8);
  }
  static __device__ __forceinline__ int* flag_of(unsigned char* sc) {
    return reinterpret_cast<int*>(sc + BN * CAP * 8 + kVals + TPQ * BN * 4 + BN * 12);
  }

  __device__ __forceinline__ float run_value(int i) const {  // value of entry i (runtime i)
    u64 c = 0ull;
#pragma unroll
    for (int j = 0; j < KS; ++j)
      if (j == i) c = run.v[j];
    return c ? comp_score(c) : kNegInf;
  }

  // One pass over rows [0, rp) of S for every query of the block.  Rows at or above the
  // running k-th value tau0 are counted first; when at most CAP of them exist (the usual case
  // once the list is full) they are appended directly.  Otherwise the query takes the full
  // path: top-KS values of the slice (independent med3 chains), the exact k-th value tau of
  // slice + running list, then rows above tau and the smallest-id rows equal to tau.
  __device__ __forceinline__ void pass(const float* S, int SR, int rp, const PassRows& pr, int q_lim, int k,
                                       unsigned char* scratch) {
    u64* cand = reinterpret_cast<u64*>(scratch);
    float* vals = reinterpret_cast<float*>(scratch + BN * CAP * 8);
    int* cnt2 = reinterpret_cast<int*>(scratch + BN * CAP * 8 + kVals);
    float* tau_s = reinterpret_cast<float*>(cnt2 + TPQ * BN);
    int* need_s = reinterpret_cast<int*>(tau_s + BN);
    int* cnt_s = need_s + BN;
    int* flag_s = cnt_s + BN;
    const int t = threadIdx.x, qq = t % BN, sub = t / BN;
    const bool active = qq < q_lim;
    const int per = rp / TPQ;
    const int r0 = sub * per;
    const float* Sq = S + qq * SR + r0;
    const int nv = pr.nvalid - r0;  // valid rows of this thread's slice: [0, nv)

    if (sub == 0) {
      tau_s[qq] = run_value(k - 1);
      cnt_s[qq] = 0;
    }
    if (t == 0) *flag_s = 0;
    lds_barrier();
    const float t0 = tau_s[qq];
    int c = 0;
    if (active) {
      for (int j = 0; j < per; j += 4) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(Sq + j);
#pragma unroll
        for (int e = 0; e < 4; ++e) c += (j + e < nv && x[e] >= t0) ? 1 : 0;
      }
    }
    int total = c;
    if constexpr (TPQ > 1) {
      cnt2[sub * BN + qq] = c;
      lds_barrier();
      total = 0;
#pragma unroll
      for (int j = 0; j < TPQ; ++j) total += cnt2[j * BN + qq];
    }
    const bool fast = total <= CAP;
    if (active && !fast) *flag_s = 1;
    lds_barrier();
    const bool any_slow = *flag_s != 0;
    if (active && fast && c > 0) {
      for (int j = 0; j < per; j += 4) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(Sq + j);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (j + e < nv && x[e] >= t0) {
            const int slot = atomicAdd(&cnt_s[qq], 1);
            cand[qq * CAP + slot] = composite(x[e], (uint32_t)pr.row(r0 + j + e));
          }
      }
    }
    if (any_slow) {  // workgroup-uniform: every thread takes the barriers below
      const bool work = active && !fast;
      ValTop<KS> L;
      L.clear();
      if (work) {
        ValTop<KS> Lp[NL];
#pragma unroll
        for (int u = 0; u < NL; ++u) Lp[u].clear();
        for (int j = 0; j < per; j += 4) {
          const f32x4 x = *reinterpret_cast<const f32x4*>(Sq + j);
#pragma unroll
          for (int e = 0; e < 4; ++e) Lp[e % NL].insert(j + e < nv ? x[e] : kNegInf);
        }
        L = Lp[0];
#pragma unroll
        for (int u = 1; u < NL; ++u)
#pragma unroll
          for (int i = 0; i < KS; ++i) L.insert(Lp[u].v[i]);
      }
      if constexpr (TPQ > 1) {
#pragma unroll
        for (int i = 0; i < KS; ++i) vals[(sub * BN + qq) * KS + i] = L.v[i];
        lds_barrier();
        if (sub == 0 && work)
          for (int j = 1; j < TPQ; ++j)
#pragma unroll
            for (int i = 0; i < KS; ++i) L.insert(vals[(j * BN + qq) * KS + i]);
      }
      if (sub == 0 && work) {
#pragma unroll
        for (int i = 0; i < KS; ++i)
          if (i < k) L.insert(run.v[i] ? comp_score(run.v[i]) : kNegInf);
        const float tau = L.at(k);
        int ngt = 0;
#pragma unroll
        for (int i = 0; i < KS; ++i) ngt += (i < k && L.v[i] > tau) ? 1 : 0;
        tau_s[qq] = tau;
        need_s[qq] = tau == kNegInf ? 0 : k - ngt;  // entries equal to tau still needed
      }
      lds_barrier();
      const float tau = tau_s[qq];
      const int need = need_s[qq];
      int neq = 0;
      if (work) {
        for (int j = 0; j < per; j += 4) {
          const f32x4 x = *reinterpret_cast<const f32x4*>(Sq + j);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (j + e < nv) {
              if (x[e] > tau) {
                const int slot = atomicAdd(&cnt_s[qq], 1);
                cand[qq * CAP + slot] = composite(x[e], (uint32_t)pr.row(r0 + j + e));
              }
              neq += x[e] == tau ? 1 : 0;
            }
          }
        }
      }
      int pre = 0;
      if constexpr (TPQ > 1) {
        cnt2[sub * BN + qq] = neq;
        lds_barrier();
        for (int j = 0; j < sub; ++j) pre += cnt2[j * BN + qq];
      }
      if (work && neq > 0 && pre < need) {
        for (int j = 0; j < per && pre < need; ++j) {
          if (j < nv && Sq[j] == tau) {
            const int slot = atomicAdd(&cnt_s[qq], 1);
            cand[qq * CAP + slot] = composite(tau, (uint32_t)pr.row(r0 + j));
            ++pre;
          }
        }
      }
    }
    lds_barrier();
    if (sub == 0 && active) {
      const int n = cnt_s[qq];
      for (int j = 0; j < n; ++j) run.insert(cand[qq * CAP + j]);
    }
    lds_barrier();
  }

  // Owner threads write the query's k best: to its chunk slot, or as the final output.
  __device__ __forceinline__ void write(const DenseArgs& a, int q0, long long chunk) const {
    const int t = threadIdx.x, qq = t % BN, sub = t / BN, q = q0 + qq;
    if (sub != 0 || q >= a.nq) return;
    if (a.n_chunks > 1) {
      u64* dst = a.partial + ((long long)q * a.n_chunks + chunk) * a.k;
#pragma unroll
      for (int i = 0; i < KS; ++i)
        if (i < a.k) dst[i] = run.v[i];
    } else {
#pragma unroll
      for (int i = 0; i < KS; ++i) {
        if (i < a.k) {
          const u64 c = run.v[i];
          a.out_ids[(long long)q * a.k + i] = c ? (long long)comp_row(c) : -1ll;
          a.out_scores[(long long)q * a.k + i] = c ? comp_score(c) : kNegInf;
        }
      }
    }
  }
};

// k <= 128.
template <int BN>
struct SelLarge {
  static constexpr int QPW = BN / kWaves;  // queries per wave (query w + 4 j)
  static constexpr int kBytes = 0;
  u64 q0[QPW], q1[QPW];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int j = 0; j < QPW; ++j) q0[j] = q1[j] = 0ull;
  }

  __device__ __forceinline__ void pass(const float* S, int SR, int rp, const PassRows& pr, int q_lim, int k,
                                       unsigned char*) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < QPW; ++j) {
      const int qq = w + kWaves * j;
      if (qq >= q_lim) continue;  // wave-uniform
      const float* Sq = S + qq * SR;
      for (int base = 0; base < rp; base += 64) {
        const int r = base + lane;
        u64 c = 0ull;
        if (r < pr.nvalid) c = composite(Sq[r], (uint32_t)pr.row(r));
        wave_offer(q0[j], q1[j], c, queue_at(q0[j], q1[j], k - 1), lane);
      }
    }
    lds_barrier();
  }

  __device__ __forceinline__ void write(const DenseArgs& a, int qbase, long long chunk) const {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < QPW; ++j) {
      const int q = qbase + w + kWaves * j;
      if (q >= a.nq) continue;
      if (a.n_chunks > 1) {
        u64* dst = a.partial + ((long long)q * a.n_chunks + chunk) * a.k;
        if (lane < a.k) dst[lane] = q0[j];
        if (lane + 64 < a.k) dst[lane + 64] = q1[j];
      } else {
        const long long o = (long long)q * a.k;
        if (lane < a.k) {
          a.out_ids[o + lane] = q0[j] ? (long long)comp_row(q0[j]) : -1ll;
          a.out_scores[o + lane] = q0[j] ? comp_score(q0[j]) : kNegInf;
        }
        if (lane + 64 < a.k) {
          a.out_ids[o + lane + 64] = q1[j] ? (long long)comp_row(q1[j]) : -1ll;
          a.out_scores[o + lane + 64] = q1[j] ? comp_score(q1[j]) : kNegInf;
        }
      }
    }
  }
};

template <int BN, int KS, int SEL, int NT>
struct SelOf {
  typedef SelSmall<BN, KS, NT> type;
};
template <int BN, int KS, int NT>
struct SelOf<BN, KS, 1, NT> {
  static_assert(NT == kThreads, "the queue selector assumes four waves");
  typedef SelLarge<BN> type;
};

// ------------------------------------------------------------------------------------
// Filtered mode (k > 16).  Every row whose score reaches the query's threshold becomes a
// candidate key in the query's global buffer; an exact selection over the buffer follows in
// select_topk_kernel.  Candidates of a query are staged in LDS (SCAP keys) and written out
// with one device-scope reservation per flush.  A staged entry holds the raw score bits and
// the row; the flush turns it into the key.  LDS: stage [BN][SCAP] | one discard slot per
// thread | flush bases [BN] | staged counts [BN].
// ------------------------------------------------------------------------------------
template <int BN>
struct SelFilter {
  static constexpr int SCAP = 32;
  static constexpr int kTrash = 256;  // threads of the kernels that use it
  static constexpr int kBytes = BN * SCAP * 8 + kTrash * 8 + BN * 8 + BN * 4;
  static __device__ __forceinline__ u64* stage(unsigned char* area) { return reinterpret_cast<u64*>(area); }
  static __device__ __forceinline__ u64* trash(unsigned char* area) { return reinterpret_cast<u64*>(area) + BN * SCAP; }
  static __device__ __forceinline__ long long* base(unsigned char* area) {
    return reinterpret_cast<long long*>(area + BN * SCAP * 8 + kTrash * 8);
  }
  static __device__ __forceinline__ int* staged(unsigned char* area) {
    return reinterpret_cast<int*>(area + BN * SCAP * 8 + kTrash * 8 + BN * 8);
  }
  __device__ __forceinline__ void init() {}
  __device__ __forceinline__ void pass(const float*, int, int, const PassRows&, int, int, unsigned char*) {}
  __device__ __forceinline__ void write(const DenseArgs&, int, long long) const {}
};
template <int BN, int KS, int NT>
struct SelOf<BN, KS, 2, NT> {
  typedef SelFilter<BN> type;
};
template <int BN, int KS, int NT>
struct SelOf<BN, KS, 4, NT> {  // filtered, many hits per tile
  typedef SelFilter<BN> type;
};

// Score dump (SEL 3): no selection; every score of the tile goes to a.dump.
struct SelDump {
  static constexpr int kBytes = 16;
  __device__ __forceinline__ void init() {}
  __device__ __forceinline__ void pass(const float*, int, int, const PassRows&, int, int, unsigned char*) {}
  __device__ __forceinline__ void write(const DenseArgs&, int, long long) const {}
};
template <int BN, int KS, int NT>
struct SelOf<BN, KS, 3, NT> {
  typedef SelDump type;
};

// acc[mi][ni][r] is the score of row tile0 + 16*MW*wave + 16*mi + 4*(lane/16) + r against
// query slot 16*ni + lane%16: four consecutive rows per lane and query, stored as one 16-byte
// write when all four exist (dump_ld is a multiple of 4).  mn / mx take the lane's running
// minimum and maximum per query slot over the rows that exist.
template <int BN, int MW, int WV>
__device__ __forceinline__ void dump_tile(const f32x4 (&acc)[MW][BN / 16], long long tile0, long long row_end,
                                          int q0, int q_lim, const DenseArgs& a, float (&mn)[BN / 16],
                                          float (&mx)[BN / 16]) {
  constexpr int NW = BN / 16;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const long long r0 = tile0 + w * MW * 16 + (lane >> 4) * 4;
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    const int n = ni * 16 + (lane & 15);
    if (n >= q_lim) continue;
    float* dst = a.dump + (long long)(q0 + n) * a.dump_ld;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi) {
      const long long row = r0 + mi * 16;
      if (row + 3 < row_end) {
        *reinterpret_cast<f32x4*>(dst + row) = acc[mi][ni];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          mn[ni] = fminf(mn[ni], acc[mi][ni][r]);
          mx[ni] = fmaxf(mx[ni], acc[mi][ni][r]);
        }
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (row + r < row_end) {
            dst[row + r] = acc[mi][ni][r];
            mn[ni] = fminf(mn[ni], acc[mi][ni][r]);
            mx[ni] = fmaxf(mx[ni], acc[mi][ni][r]);
          }
      }
    }
  }
}

// Staged entry -> key.
__device__ __forceinline__ u64 staged_key(u64 e) { return composite(__uint_as_float((uint32_t)(e >> 32)), (uint32_t)e); }

// Owner thread of query slot n: append its staged keys (a count beyond SCAP means the rest
// already went out directly) to the global buffer, with no barrier (a mid-chunk flush).
template <int BN>
__device__ __forceinline__ void filt_flush_owner(int n, int q, unsigned char* area, const DenseArgs& a) {
  constexpr int SCAP = SelFilter<BN>::SCAP;
  const u64* stage = SelFilter<BN>::stage(area);
  int* staged = SelFilter<BN>::staged(area);
  const int c = min(staged[n], SCAP);
  if (c == 0) return;
  const long long g = atomicAdd(a.ccnt + q, c);
  u64* dst = a.cbuf + (long long)q * a.cap;
  for (int j = 0; j < c; ++j)
    if (g + j < a.cap) dst[g + j] = staged_key(stage[n * SCAP + j]);
  staged[n] = 0;
}

// Flush of every staged key at the end of a chunk: the owner threads reserve their slots in
// the global buffers with one device-scope atomic each, all at once; after a barrier every
// thread copies staged keys, consecutive threads taking consecutive keys of a query.
template <int BN, int NT>
__device__ __forceinline__ void filt_flush(unsigned char* area, int q0, int q_lim, const DenseArgs& a) {
  constexpr int SCAP = SelFilter<BN>::SCAP;
  const u64* stage = SelFilter<BN>::stage(area);
  long long* base = SelFilter<BN>::base(area);
  int* staged = SelFilter<BN>::staged(area);
  const int tid = threadIdx.x;
  if (tid < BN) {
    const int c = min(staged[tid], SCAP);
    base[tid] = tid < q_lim && c > 0 ? (long long)atomicAdd(a.ccnt + q0 + tid, c) : -1ll;
  }
  lds_barrier();
#pragma unroll 4
  for (int i = tid; i < BN * SCAP; i += NT) {
    const int n = i / SCAP, j = i % SCAP;
    const long long g = base[n] + j;
    if (base[n] >= 0 && j < min(staged[n], SCAP) && g < a.cap) a.cbuf[(long long)(q0 + n) * a.cap + g] = staged_key(stage[i]);
  }
}

// Hits of one tile, few of them (most tiles of a long chunk have none): a lane compares the
// maximum of its MW*4 scores of a query with the threshold and, on a hit, counts them,
// reserves that many stage slots with one LDS atomic and writes them; hits past the stage's
// end go straight to the global buffer under one device-scope reservation.  FULL: the tile
// lies inside the chunk (no row-limit test).
template <bool FULL, int BN, int MW>
__device__ __forceinline__ void filt_collect_sparse(const f32x4 (&acc)[MW][BN / 16], const float (&th)[BN / 16],
                                                    unsigned char* area, long long tile0, int row0, int lim, int q0,
                                                    const DenseArgs& a) {
  constexpr int NW = BN / 16;
  constexpr int SCAP = SelFilter<BN>::SCAP;
  u64* stage = SelFilter<BN>::stage(area);
  int* staged = SelFilter<BN>::staged(area);
  const int lane = threadIdx.x & 63;
  const uint32_t row_l = (uint32_t)(tile0 + row0);
  auto ok = [&](int mi, int r) { return FULL || mi * 16 + r < lim; };
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    float m = kNegInf;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) m = __builtin_fmaxf(m, ok(mi, r) ? acc[mi][ni][r] : kNegInf);
    if (!(m >= th[ni])) continue;
    int c = 0;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) c += (ok(mi, r) && acc[mi][ni][r] >= th[ni]) ? 1 : 0;
    const int n = ni * 16 + (lane & 15);
    const int pos = atomicAdd(&staged[n], c);
    const int in_stage = max(0, min(c, SCAP - pos));
    const long long g = in_stage < c ? atomicAdd(a.ccnt + q0 + n, c - in_stage) : 0ll;
    u64* dst_g = a.cbuf + (long long)(q0 + n) * a.cap;
    int h = 0;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x = acc[mi][ni][r];
        if (ok(mi, r) && x >= th[ni]) {
          const uint32_t row = row_l + (uint32_t)(mi * 16 + r);
          if (h < in_stage) {
            stage[n * SCAP + pos + h] = ((u64)__float_as_uint(x) << 32) | (u64)row;
          } else {
            const long long j = g + (h - in_stage);
            if (j < a.cap) dst_g[j] = composite(x, row);
          }
          ++h;
        }
      }
  }
}

// Hits of one tile, many of them.  Each lane first forms, for every query slot, the mask of
// its MW*4 scores that reach the threshold, then reserves that many stage slots per slot with
// hits (one LDS atomic each, all issued before the first result is used), then stores every
// score of a slot with hits without a branch: a hit to its stage slot, any other score to the
// thread's discard slot.  Hits past the stage's end (rare) go straight to the global buffer
// under one device-scope reservation.  FULL: the tile lies inside the chunk (no row-limit
// test).
template <bool FULL, int BN, int MW>
__device__ __forceinline__ void filt_collect_dense(const f32x4 (&acc)[MW][BN / 16], const float (&th)[BN / 16],
                                             unsigned char* area, long long tile0, int row0, int lim, int q0,
                                             const DenseArgs& a) {
  constexpr int NW = BN / 16;
  constexpr int SCAP = SelFilter<BN>::SCAP;
  static_assert(MW * 4 <= 32, "a lane's scores of a query slot fit one mask");
  u64* stage = SelFilter<BN>::stage(area);
  int* staged = SelFilter<BN>::staged(area);
  u64* trash = SelFilter<BN>::trash(area) + threadIdx.x;
  const int lane = threadIdx.x & 63;
  auto ok = [&](int mi, int r) { return FULL || mi * 16 + r < lim; };
  // a slot's mask is formed only when the maximum of its scores reaches the threshold (after
  // the first tiles of a long chunk hits are rare, and a wave then skips whole slots)
  uint32_t bits[NW];
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    float m = kNegInf;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) m = __builtin_fmaxf(m, ok(mi, r) ? acc[mi][ni][r] : kNegInf);
    uint32_t b = 0u;
    if (m >= th[ni]) {
#pragma unroll
      for (int mi = 0; mi < MW; ++mi)
#pragma unroll
        for (int r = 0; r < 4; ++r) b |= (ok(mi, r) && acc[mi][ni][r] >= th[ni] ? 1u : 0u) << (mi * 4 + r);
    }
    bits[ni] = b;
  }
  int pos[NW];
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    const int c = __popc(bits[ni]);
    pos[ni] = c ? atomicAdd(&staged[ni * 16 + (lane & 15)], c) : 0;
  }
  const uint32_t row_l = (uint32_t)(tile0 + row0);
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    const uint32_t b = bits[ni];
    if (b == 0u) continue;  // a slot no lane of the wave hits is skipped by the whole wave
    const int c = __popc(b), n = ni * 16 + (lane & 15);
    const int in_stage = max(0, min(c, SCAP - pos[ni]));
    u64* st = stage + n * SCAP + pos[ni];
    int h = 0;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int hit = (int)((b >> (mi * 4 + r)) & 1u);
        u64* dst = hit && h < in_stage ? st + h : trash;
        *dst = ((u64)__float_as_uint(acc[mi][ni][r]) << 32) | (u64)(row_l + (uint32_t)(mi * 16 + r));
        h += hit;
      }
    if (in_stage < c) {  // the lane's hits past the stage
      const long long g = atomicAdd(a.ccnt + q0 + n, c - in_stage);
      u64* dst_g = a.cbuf + (long long)(q0 + n) * a.cap;
      int hh = 0;
#pragma unroll
      for (int mi = 0; mi < MW; ++mi)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if ((b >> (mi * 4 + r)) & 1u) {
            const long long jg = g + (hh - in_stage);
            if (hh >= in_stage && jg < a.cap) dst_g[jg] = composite(acc[mi][ni][r], row_l + (uint32_t)(mi * 16 + r));
            ++hh;
          }
    }
  }
}

// First level (no threshold): every row of [0, n_rows) is a candidate, so each score goes to
// the slot of its row in the query's buffer; no counting, no atomics, no barrier.  The
// buffer holds at least n_rows keys at this level.
template <int BN, int MW, int WV>
__device__ __forceinline__ void filt_all_tile(const f32x4 (&acc)[MW][BN / 16], long long tile0, long long row_end,
                                              int q0, int q_lim, const DenseArgs& a) {
  constexpr int NW = BN / 16;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const long long r0 = tile0 + w * MW * 16 + (lane >> 4) * 4;
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    const int n = ni * 16 + (lane & 15);
    if (n >= q_lim) continue;
    u64* dst = a.cbuf + (long long)(q0 + n) * a.cap;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const long long row = r0 + mi * 16 + r;
        if (row < row_end) dst[row] = composite(acc[mi][ni][r], (uint32_t)row);
      }
  }
}

// acc[mi][ni][r] = score of row tile0 + 16*MW*wave + 16*mi + 4*(lane/16) + r against query
// slot 16*ni + lane%16; th[ni] its threshold (+inf for slots past the batch).  One barrier;
// then the chunk's last tile flushes every stage together, and after an earlier tile the
// owners of stages at least half full flush theirs.  The stage is next written in the
// following tile's selection, after a barrier inside that tile's main loop.
template <bool DH, int BN, int MW, int WV>
__device__ __forceinline__ void filt_tile(const f32x4 (&acc)[MW][BN / 16], const float (&th)[BN / 16],
                                          unsigned char* area, long long tile0, long long row_end, int q0, int q_lim,
                                          bool last, bool check, const DenseArgs& a) {
  constexpr int SCAP = SelFilter<BN>::SCAP;
  constexpr int TR = WV * MW * 16;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int row0 = w * MW * 16 + (lane >> 4) * 4;
  const int lim = (int)(row_end - tile0) - row0;
  if constexpr (DH) {
    if (tile0 + TR <= row_end)  // workgroup-uniform
      filt_collect_dense<true, BN, MW>(acc, th, area, tile0, row0, 0, q0, a);
    else
      filt_collect_dense<false, BN, MW>(acc, th, area, tile0, row0, lim, q0, a);
  } else {
    if (tile0 + TR <= row_end)
      filt_collect_sparse<true, BN, MW>(acc, th, area, tile0, row0, 0, q0, a);
    else
      filt_collect_sparse<false, BN, MW>(acc, th, area, tile0, row0, lim, q0, a);
  }
  // The stage is looked at (and flushed) only on check tiles; in between it fills, and hits
  // past its capacity go straight to the global buffer (filt_collect_*), so no barrier is needed.
  if (!check && !last) return;  // workgroup-uniform
  lds_barrier();
  if (last)  // workgroup-uniform
    filt_flush<BN, WV * 64>(area, q0, q_lim, a);
  else if (tid < BN && SelFilter<BN>::staged(area)[tid] >= SCAP / 2)
    filt_flush_owner<BN>(tid, q0 + tid, area, a);
}

// ------------------------------------------------------------------------------------
// Selection straight from the MFMA accumulators (k <= 16).  acc[mi][ni][r] is the score of
// row tile0 + 16*MW*wave + 16*mi + 4*(lane/16) + r against query 16*ni + lane%16 of the
// block.  Each lane's MW*4 values of a query form one group; the M best values of every
// group are actual, distinct scores, so the k-th largest of them together with the running
// list is a lower bound tau of the k-th best score so far.  Only scores >= tau (a handful per
// query) go to LDS as candidates and the owner thread inserts them into its running list.
// Returns false, with the running lists untouched, when some query has more than CAP
// candidates (many equal scores); the caller then takes the exact LDS path.
// ------------------------------------------------------------------------------------
template <int BN, int MW, int KS, int WV, typename Sel>
__device__ __forceinline__ bool reg_epilogue(const f32x4 (&acc)[MW][BN / 16], Sel& sel, float* gv,
                                             unsigned char* scratch, long long tile0, long long row_end, int q_lim,
                                             int k) {
  constexpr int NW = BN / 16;
  constexpr int M = KS <= 5 ? 1 : (KS <= 8 ? 2 : 4);  // values kept per group
  constexpr int NG = WV * 4 * M;                      // group values per query
  constexpr int CAP = Sel::CAP;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // candidates as (score bits, row offset in the tile), in the candidate area of the selector
  uint2* cand = reinterpret_cast<uint2*>(Sel::cand_of(scratch));
  float* thr = Sel::tau_of(scratch);
  int* cnt = Sel::cnt_of(scratch);
  int* flag = Sel::flag_of(scratch);
  constexpr int TR = WV * MW * 16;
  const int row0 = w * MW * 16 + (lane >> 4) * 4;  // tile offset of this lane's value (0, r = 0)
  // element (mi, r) of this lane is a valid row iff 16*mi + r < lim
  const int lim = (int)min((long long)TR, row_end - tile0) - row0;
  const int g = w * 4 + (lane >> 4);

#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    ValTop<M> t;
    t.clear();
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) t.insert(mi * 16 + r < lim ? acc[mi][ni][r] : kNegInf);
#pragma unroll
    for (int j = 0; j < M; ++j) gv[(g * M + j) * BN + ni * 16 + (lane & 15)] = t.v[j];
  }
  lds_barrier();
  if (tid < BN) {
    float tau = __builtin_inff();  // queries past the batch take no candidates
    if (tid < q_lim) {
      ValTop<KS> L;
      L.clear();
      for (int j = 0; j < NG; ++j) L.insert(gv[j * BN + tid]);
#pragma unroll
      for (int i = 0; i < KS; ++i)
        if (i < k && sel.run.v[i]) L.insert(comp_score(sel.run.v[i]));
      tau = L.at(k);
    }
    thr[tid] = tau;
    cnt[tid] = 0;
  }
  if (tid == 0) *flag = 0;
  lds_barrier();
  // Count first, reserve once per (lane, query), then write: one LDS atomic per query
  // fragment instead of one per candidate.
  float th[NW];
  int c[NW], base[NW];
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    th[ni] = thr[ni * 16 + (lane & 15)];
    int cc = 0;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) cc += (mi * 16 + r < lim && acc[mi][ni][r] >= th[ni]) ? 1 : 0;
    c[ni] = cc;
  }
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) base[ni] = c[ni] ? atomicAdd(&cnt[ni * 16 + (lane & 15)], c[ni]) : 0;
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    if (c[ni] == 0) continue;
    if (base[ni] + c[ni] > CAP) {
      *flag = 1;
      continue;
    }
    uint2* dst = cand + (ni * 16 + (lane & 15)) * CAP;
    int j = base[ni];
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x = acc[mi][ni][r];
        if (mi * 16 + r < lim && x >= th[ni]) {
          dst[j] = make_uint2(__float_as_uint(x), (unsigned)(row0 + mi * 16 + r));
          ++j;
        }
      }
  }
  lds_barrier();
  if (*flag) return false;
  if (tid < q_lim) {
    const int n = cnt[tid];
    for (int j = 0; j < n; ++j) {
      const uint2 e = cand[tid * CAP + j];
      sel.run.insert(composite(__uint_as_float(e.x), (uint32_t)(tile0 + e.y)));
    }
  }
  return true;
}

// ------------------------------------------------------------------------------------
// Selection against the running threshold (k <= 16 except the larger k <= 5 kernels; every tile
// after a chunk's first).
// thr[n] holds the k-th best score of query slot n's running list (-inf while the list is
// short, +inf past the batch); only a score reaching it can still enter the list.  A lane
// first compares the maximum of its MW*4 scores of each query with the threshold, so a tile
// with nothing new costs a few dozen instructions per lane and one barrier.  Hits are
// appended to the query's candidate list (count, reserve once per lane and query, write);
// the owner threads insert them and raise thr.  Returns false, with the lists untouched, when
// some query has more than CAP hits in the tile; the caller then takes the group path.
// ------------------------------------------------------------------------------------
// Hits of this lane against the thresholds: count, reserve once per query, write.  FULL: the
// tile lies inside the chunk, so no row needs the row-limit test.
template <bool FULL, int BN, int MW, int CAP>
__device__ __forceinline__ void thr_collect(const f32x4 (&acc)[MW][BN / 16], const float* thr, int* cnt, int* flag,
                                            uint2* cand, int row0, int lim) {
  constexpr int NW = BN / 16;
  const int lane = threadIdx.x & 63;
  auto ok = [&](int mi, int r) { return FULL || mi * 16 + r < lim; };
  // the thresholds of this lane's query slots, read together (one wait), and the maxima
  float th[NW], mx[NW];
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) th[ni] = thr[ni * 16 + (lane & 15)];
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    float m = kNegInf;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) m = __builtin_fmaxf(m, ok(mi, r) ? acc[mi][ni][r] : kNegInf);
    mx[ni] = m;
  }
  bool any = false;
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) any |= mx[ni] >= th[ni];
  if (__ballot(any) == 0ull) return;  // wave-uniform: no score of this wave reaches its threshold
  int c[NW];
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    int cc = 0;
    if (mx[ni] >= th[ni]) {
#pragma unroll
      for (int mi = 0; mi < MW; ++mi)
#pragma unroll
        for (int r = 0; r < 4; ++r) cc += (ok(mi, r) && acc[mi][ni][r] >= th[ni]) ? 1 : 0;
    }
    c[ni] = cc;
  }
  int base[NW];
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) base[ni] = c[ni] ? atomicAdd(&cnt[ni * 16 + (lane & 15)], c[ni]) : 0;
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    if (c[ni] == 0) continue;
    if (base[ni] + c[ni] > CAP) {
      *flag = 1;
      continue;
    }
    const int n = ni * 16 + (lane & 15);
    uint2* dst = cand + n * CAP;
    int j = base[ni];
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x = acc[mi][ni][r];
        if (ok(mi, r) && x >= th[ni]) {
          dst[j] = make_uint2(__float_as_uint(x), (unsigned)(row0 + mi * 16 + r));
          ++j;
        }
      }
  }
}

template <int BN, int MW, int WV, typename Sel>
__device__ __forceinline__ bool thr_epilogue(const f32x4 (&acc)[MW][BN / 16], Sel& sel, unsigned char* scratch,
                                             long long tile0, long long row_end, int q_lim, int k) {
  constexpr int CAP = Sel::CAP;
  constexpr int TR = WV * MW * 16;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  uint2* cand = reinterpret_cast<uint2*>(Sel::cand_of(scratch));
  float* thr = Sel::tau_of(scratch);
  int* cnt = Sel::cnt_of(scratch);
  int* flag = Sel::flag_of(scratch) + 1;  // a word of its own: the group path uses the first
  const int row0 = w * MW * 16 + (lane >> 4) * 4;
  if (tile0 + TR <= row_end)  // workgroup-uniform
    thr_collect<true, BN, MW, CAP>(acc, thr, cnt, flag, cand, row0, 0);
  else
    thr_collect<false, BN, MW, CAP>(acc, thr, cnt, flag, cand, row0, (int)(row_end - tile0) - row0);
  lds_barrier();
  if (*flag) {  // uniform; the group path resets cnt, and thr_reset thr and flag after it
    lds_barrier();
    return false;
  }
  if (tid < q_lim) {
    const int n = cnt[tid];
    if (n > 0) {
      for (int j = 0; j < n; ++j) {
        const uint2 e = cand[tid * CAP + j];
        sel.run.insert(composite(__uint_as_float(e.x), (uint32_t)(tile0 + e.y)));
      }
      cnt[tid] = 0;
      thr[tid] = sel.run_value(k - 1);
    }
  }
  // thr and cnt are next read in the following tile's selection, after the barriers of its
  // super-steps
  return true;
}

// After a tile that took the group path (or the LDS passes): owners restore the running
// threshold and an empty candidate list.  After the last barrier of that path a thread reads
// only its own query's thr and cnt, and the fast path's overflow word was last read before
// the barrier that preceded the group path.
template <typename Sel>
__device__ __forceinline__ void thr_reset(const Sel& sel, unsigned char* scratch, int q_lim, int k, int bn) {
  const int tid = threadIdx.x;
  if (tid < bn) {
    Sel::tau_of(scratch)[tid] = tid < q_lim ? sel.run_value(k - 1) : __builtin_inff();
    Sel::cnt_of(scratch)[tid] = 0;
  }
  if (tid == 0) Sel::flag_of(scratch)[1] = 0;
}

// ------------------------------------------------------------------------------------
// k <= 5: the same lower bound tau from the group maxima, but the groups themselves are
// handed over: a lane whose maximum for a query reaches tau (at most k such groups per
// query, barring ties) copies its MW*4 scores of that query to one of SLOTS blocks in LDS,
// and the owner thread takes every score >= tau from its query's blocks.  Returns false,
// with the running lists untouched, when a query has more than SLOTS such groups.
// ------------------------------------------------------------------------------------
template <int MW, int BN>
struct BlockArea {
  static constexpr int SLOTS = 7;
  static constexpr int VALS = MW * 4;              // scores per block
  static constexpr int QSTR = SLOTS * VALS + 4;    // floats per query; the pad spreads banks
  static constexpr int kBytes = BN * QSTR * 4 + BN * 4;
};

template <int BN, int MW, int WV, typename Sel>
__device__ __forceinline__ bool blk_epilogue(const f32x4 (&acc)[MW][BN / 16], Sel& sel, unsigned char* area,
                                             unsigned char* scratch, long long tile0, long long row_end, int q_lim,
                                             int k, bool split) {
  constexpr int NW = BN / 16;
  constexpr int KS = 5;
  constexpr int NG = WV * 4;              // groups (lanes) per query
  using B = BlockArea<MW, BN>;
  constexpr int SLOTS = B::SLOTS, VALS = B::VALS, QSTR = B::QSTR;
  float* blk = reinterpret_cast<float*>(area);                      // [BN][QSTR]: SLOTS x VALS
  unsigned* gmask = reinterpret_cast<unsigned*>(area + BN * QSTR * 4);  // [BN] active groups
  float* gmax = reinterpret_cast<float*>(Sel::cand_of(scratch));    // [NG][BN]
  float* thr = Sel::tau_of(scratch);
  int* cnt = Sel::cnt_of(scratch);
  int* flag = Sel::flag_of(scratch);
  constexpr int TR = WV * MW * 16;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = w * 4 + (lane >> 4);
  const int lim = (int)min((long long)TR, row_end - tile0) - (w * MW * 16 + (lane >> 4) * 4);

  // 1. group maxima
  float lmax[NW];
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    float m = kNegInf;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) m = __builtin_fmaxf(m, mi * 16 + r < lim ? acc[mi][ni][r] : kNegInf);
    lmax[ni] = m;
    gmax[g * BN + ni * 16 + (lane & 15)] = m;
  }
  if (tid == 0) *flag = 0;
  lds_barrier();
  // 2. owners: tau, and the groups whose maximum reaches it (slot = rank among them)
  if (tid < BN) {
    float tau = __builtin_inff();  // queries past the batch take no candidates
    unsigned mask = 0;
    if (tid < q_lim) {
      float gm[NG];
#pragma unroll
      for (int j = 0; j < NG; ++j) gm[j] = gmax[j * BN + tid];
      ValTop<KS> L;
      L.clear();
#pragma unroll
      for (int j = 0; j < NG; ++j) L.insert(gm[j]);
#pragma unroll
      for (int i = 0; i < KS; ++i)
        if (i < k && sel.run.v[i]) L.insert(comp_score(sel.run.v[i]));
      tau = L.at(k);
#pragma unroll
      for (int j = 0; j < NG; ++j) mask |= (gm[j] >= tau && gm[j] > kNegInf) ? 1u << j : 0u;
      if (__builtin_popcount(mask) > SLOTS) *flag = 1;
    }
    thr[tid] = tau;
    gmask[tid] = mask;
    cnt[tid] = 0;
  }
  lds_barrier();
  if (*flag) return false;
  // 3. active groups copy their scores of the query to the block of their rank
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    const int n = ni * 16 + (lane & 15);
    const unsigned mask = gmask[n];
    if ((mask >> g) & 1u) {
      const int slot = __builtin_popcount(mask & ((1u << g) - 1u));
      float* dst = blk + n * QSTR + slot * VALS;
#pragma unroll
      for (int mi = 0; mi < MW; ++mi) {
        f32x4 v = acc[mi][ni];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = mi * 16 + r < lim ? v[r] : kNegInf;
        *reinterpret_cast<f32x4*>(dst + mi * 4) = v;
      }
    }
  }
  lds_barrier();
  // 4. the scores >= tau of the query's blocks go into its list: a mask of the hits of a block
  // (one per active group, so usually a single bit), then one insertion per set bit with the
  // score re-read at its offset.  The owner (sub 0) does this alone, except with split (a
  // chunk's first tile, where most hits fall): then the query's two threads take alternate
  // blocks, sub 1 into its own (otherwise empty) list, which it hands to the owner through LDS.
  constexpr int SP = WV * 64 / BN >= 2 ? 2 : 1;  // threads sharing a query's blocks
  const int qq = tid % BN, sub = tid / BN;
  const int sp = split ? SP : 1;
  if (qq < q_lim && sub < sp) {
    const float tau = thr[qq];
    int rank = 0;
    for (unsigned mm = gmask[qq]; mm; mm &= mm - 1, ++rank) {
      if (sp == 2 && (rank & 1) != sub) continue;
      const int gg = __builtin_ctz(mm);
      const long long r0 = tile0 + (gg >> 2) * MW * 16 + (gg & 3) * 4;
      const float* src = blk + qq * QSTR + rank * VALS;
      unsigned hm = 0;
#pragma unroll
      for (int mi = 0; mi < MW; ++mi) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(src + mi * 4);
#pragma unroll
        for (int r = 0; r < 4; ++r) hm |= (v[r] >= tau && v[r] > kNegInf) ? 1u << (mi * 4 + r) : 0u;
      }
      for (; hm; hm &= hm - 1) {
        const int pp = __builtin_ctz(hm);
        sel.run.insert(composite(src[pp], (uint32_t)(r0 + (pp >> 2) * 16 + (pp & 3))));
      }
    }
  }
  if (SP == 2 && split) {
    u64* hand = Sel::cand_of(scratch);  // [BN][KS]; the group maxima there are consumed
    if (sub == 1 && qq < q_lim) {
#pragma unroll
      for (int i = 0; i < KS; ++i) hand[qq * KS + i] = sel.run.v[i];
      sel.run.clear();
    }
    lds_barrier();
    if (sub == 0 && qq < q_lim) {
#pragma unroll
      for (int i = 0; i < KS; ++i) {
        const u64 c = hand[qq * KS + i];
        if (c) sel.run.insert(c);
      }
    }
  }
  return true;
}

// ------------------------------------------------------------------------------------
// k <= 8, group path: tau = the k-th largest of the lanes' group maxima and the running list
// is a lower bound of the k-th best score (k distinct rows reach it), so the query's top k
// lies among its running entries and the tile's scores >= tau.  Every lane writes its scores
// >= tau to the query's candidate list in LDS (slot-major, [CAPR][BN]; count, reserve once,
// write); the query's owner thread then reads all of them at once, with every load in flight
// before the first insertion, and inserts them into its running list.  Returns false, with
// the running lists untouched, when a query has more than CAPR candidates (many equal scores
// at tau).
// ------------------------------------------------------------------------------------
template <int BN, int WV>
struct RankArea {
  static constexpr int NG = WV * 4;  // groups (lane quarters of a wave) per query
  static constexpr int CAPR = 16;
  static constexpr int kBytes = NG * BN * 4 + CAPR * BN * 8;
};

template <int BN, int MW, int KS, int WV, typename Sel>
__device__ __forceinline__ bool rank_epilogue(const f32x4 (&acc)[MW][BN / 16], Sel& sel, unsigned char* area,
                                              unsigned char* scratch, long long tile0, long long row_end, int q_lim,
                                              int k) {
  constexpr int NW = BN / 16;
  using RA = RankArea<BN, WV>;
  constexpr int NG = RA::NG, CAPR = RA::CAPR;
  static_assert(KS <= 8, "the group maxima bound the k-th score for small k");
  float* gmax = reinterpret_cast<float*>(area);                    // [NG][BN]
  u64* cand = reinterpret_cast<u64*>(area + NG * BN * 4);          // [CAPR][BN]
  float* thr = Sel::tau_of(scratch);
  int* cnt = Sel::cnt_of(scratch);
  int* flag = Sel::flag_of(scratch);
  constexpr int TR = WV * MW * 16;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = w * 4 + (lane >> 4);
  const int row0 = w * MW * 16 + (lane >> 4) * 4;  // tile offset of this lane's value (0, r = 0)
  // element (mi, r) of this lane is a valid row iff 16 mi + r < lim
  const int lim = (int)min((long long)TR, row_end - tile0) - row0;

  // 1. group maxima
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    float m = kNegInf;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) m = __builtin_fmaxf(m, mi * 16 + r < lim ? acc[mi][ni][r] : kNegInf);
    gmax[g * BN + ni * 16 + (lane & 15)] = m;
  }
  if (tid == 0) *flag = 0;
  lds_barrier();
  // 2. owners: tau
  if (tid < BN) {
    float tau = __builtin_inff();  // queries past the batch take no candidates
    if (tid < q_lim) {
      float gm[NG];
#pragma unroll
      for (int j = 0; j < NG; ++j) gm[j] = gmax[j * BN + tid];
      ValTop<KS> L;
      L.clear();
#pragma unroll
      for (int j = 0; j < NG; ++j) L.insert(gm[j]);
#pragma unroll
      for (int i = 0; i < KS; ++i)
        if (i < k && sel.run.v[i]) L.insert(comp_score(sel.run.v[i]));
      tau = L.at(k);
    }
    thr[tid] = tau;
    cnt[tid] = 0;
  }
  lds_barrier();
  // 3. this lane's scores reaching tau: count, reserve once per query, write
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    const int n = ni * 16 + (lane & 15);
    const float th = thr[n];
    int c = 0;
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) c += (mi * 16 + r < lim && acc[mi][ni][r] >= th) ? 1 : 0;
    if (c == 0) continue;
    int j = atomicAdd(&cnt[n], c);
    if (j + c > CAPR) {
      *flag = 1;
      continue;
    }
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x = acc[mi][ni][r];
        if (mi * 16 + r < lim && x >= th) cand[(j++) * BN + n] = composite(x, (uint32_t)(tile0 + row0 + mi * 16 + r));
      }
  }
  lds_barrier();
  if (*flag) return false;
  // 4. owners: every candidate read at once, then inserted (a wave stops at its largest count)
  if (tid < q_lim) {
    const int n = cnt[tid];
    u64 c[CAPR];
#pragma unroll
    for (int j = 0; j < CAPR; ++j) c[j] = j < n ? cand[j * BN + tid] : 0ull;
#pragma unroll
    for (int j = 0; j < CAPR; ++j)
      if (c[j]) sel.run.insert(c[j]);
  }
  return true;
}

// ------------------------------------------------------------------------------------
// First tile of a chunk in the 16-query, 64-row-tile kernels with k <= KS = 16: the
// running lists are still empty, so each query's k best rows of the tile are found by exact
// ranks instead of insertions.  Every score goes to LDS as its composite (query q's row i at
// q * 64 + (i ^ 2q), which puts the 16 queries' entries of one row in distinct banks); thread
// t ranks rows 4s .. 4s + 3 of query q = t % 16 (s = t / 16) against the query's valid rows
// (composites are unique, so the ranks are a permutation), writes those of rank below k to
// the query's candidate slots in rank order, and the owner copies them into its list.
// ------------------------------------------------------------------------------------
template <int KS, int WV, typename Sel>
__device__ __forceinline__ void first_tile_rank(const f32x4 (&acc)[1][1], Sel& sel, unsigned char* scratch,
                                                long long tile0, long long row_end, int q_lim, int k) {
  constexpr int BN = 16, TR = WV * 16, CAP = Sel::CAP;
  static_assert(TR == 64 && WV * 64 == BN * TR / 4, "16 threads per query, four rows each");
  static_assert(Sel::kVals >= BN * TR * 8 && CAP >= KS, "scratch areas");
  u64* lists = Sel::cand_of(scratch);                                   // [BN][CAP]
  u64* keys = reinterpret_cast<u64*>(scratch + BN * CAP * 8);           // [BN][TR], swizzled
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nvalid = (int)min((long long)TR, row_end - tile0);
  {
    const int n = lane & 15, row0 = w * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      keys[n * TR + ((row0 + r) ^ (2 * n))] = composite(acc[0][0][r], (uint32_t)(tile0 + row0 + r));
  }
  lds_barrier();
  const int q = tid & 15, s = tid >> 4;
  const u64* kq = keys + q * TR;
  u64 mine[4];
  int rank[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    mine[e] = kq[(4 * s + e) ^ (2 * q)];
    rank[e] = 0;
  }
#pragma unroll 16
  for (int i = 0; i < TR; ++i) {
    const u64 x = kq[i ^ (2 * q)];
    const bool v = i < nvalid;
#pragma unroll
    for (int e = 0; e < 4; ++e) rank[e] += (v && x > mine[e]) ? 1 : 0;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (4 * s + e < nvalid && rank[e] < k) lists[q * CAP + rank[e]] = mine[e];
  lds_barrier();
  if (tid < q_lim) {
    const int nv = min(k, nvalid);
#pragma unroll
    for (int i = 0; i < KS; ++i) sel.run.v[i] = i < nv ? lists[tid * CAP + i] : 0ull;
  }
}

// ------------------------------------------------------------------------------------
// bf16 / fp16 MFMA kernel.  Four waves split a tile of TR = 4*MW*16 rows (each wave owns
// MW distinct 16-row subtiles) and share a block of BN = NW*16 queries.  A k-step is one
// MFMA depth (32 dimensions); four k-steps form a super-step of 128 dimensions.
//  - Row fragments go global -> VGPRs directly in MFMA A-operand layout (each wave reads
//    only its own rows); a register ring of RS k-steps keeps RS - 1 of them in flight.
//    Every k-step issues the same loads (past the end they repeat the last k-step), so
//    the compiler's load counters stay exact and no wait drains the ring.
//  - The query block of a super-step (BN x 128 dimensions) is loaded one super-step
//    ahead into VGPRs, written to one of two LDS slots at the end of the previous
//    super-step, and read by every wave as B operands, one k-step ahead of its MFMAs.
//    One barrier per super-step.  With QR > 0 (d <= 128 QR) every super-step of the
//    queries instead stays resident in its own LDS slot, loaded once before the first
//    tile, and the loop has one barrier per tile.
//  - After the last k-step of a tile the scores sit in the accumulators; the register
//    epilogue (or, when it declines, G passes through an LDS score tile) updates the
//    running top-k of each query, or (SEL 2) the filtered mode collects the scores that
//    reach the query's threshold.
// ------------------------------------------------------------------------------------
#ifdef OPRAG_DENSE_ILP
}  // namespace: the instances below have external linkage (the kernel table refers to them)
#define OPRAG_DENSE_KERNEL dense_mfma_kernel_ilp
#else
#define OPRAG_DENSE_KERNEL dense_mfma_kernel
#endif
template <int DT, int NW, int MW, int RS, int G, int KS, int SEL, int WV, int QR>
__global__ __launch_bounds__(WV * 64) void OPRAG_DENSE_KERNEL(DenseArgs a) {
  if (a.gate != nullptr && *a.gate == 0) return;  // a repair launch with nothing to repair
  using M = Mfma<DT>;
  using V = typename M::V;
  using T = typename M::T;
  constexpr int BN = NW * 16;
  constexpr int NT = WV * 64;                  // threads
  constexpr int TR = WV * MW * 16;
  constexpr int KC = 32;                        // dimensions per k-step
  constexpr int SK = 128;                       // dimensions per super-step
  constexpr int PX = RS - 1;
  static_assert(RS == 4 || RS == 8 || RS == 16, "ring of whole super-steps");
  constexpr int BODY = RS;                      // k-steps per loop iteration; divides d / 32
  constexpr int QSLOT = BN * SK * 2;            // bytes: query row n at n * 256
  constexpr int QPT = BN * SK * 2 / 16 / NT;   // 16-byte query pieces per thread
  static_assert(QPT * NT * 16 == QSLOT, "query pieces");
  constexpr int MWP = MW / G;                   // subtile rows per wave per fallback pass
  constexpr int RP = WV * MWP * 16;             // rows per fallback pass
  constexpr int SR = RP + 4;                    // S row stride (floats)
  using Sel = typename SelOf<BN, KS, SEL, NT>::type;
  // QR > 0: all d / 128 <= QR super-steps of the block's queries stay resident in LDS (loaded
  // once), so the main loop has no query staging and no barrier.  Otherwise two slots
  // alternate, one super-step ahead.
  constexpr int QBYTES = (QR > 0 ? QR : 2) * QSLOT;
  static_assert(QR == 0 || SEL == 0 || SEL == 2 || SEL == 4, "resident queries: lists or filtered selection");
  constexpr bool kFilt = SEL == 2 || SEL == 4;  // filtered: 4 is the variant for many hits per tile
  constexpr int kFiltCheck = 32;  // SEL 2: tiles between looks at the stage (a power of two)
  // k <= 5: the small-tile kernels take the one-pass rank epilogue (and the running-threshold
  // test for later tiles); the 128-query kernel keeps the block epilogue on every tile, which
  // leaves its main loop the register budget it is scheduled for.
  constexpr bool kBlk = SEL == 0 && KS == 5 && NW * MW > 2;
  constexpr bool kRank = SEL == 0 && KS == 5 && !kBlk;
  // 9 <= k <= 16 on 16-query, 64-row tiles: a chunk's first tile by exact ranks (the group path
  // keeps four values per group for KS 16, and its owners' insertions took longer; with KS 8 the
  // group path is the faster one)
  constexpr bool kTileRank = SEL == 0 && KS == 16 && NW == 1 && MW == 1 && WV == 4;
  constexpr int SB0 = SEL >= 2 ? 0 : BN * SR * 4;
  constexpr int SBYTES = kBlk && BlockArea<MW, BN>::kBytes > SB0   ? BlockArea<MW, BN>::kBytes
                         : kRank && RankArea<BN, WV>::kBytes > SB0 ? RankArea<BN, WV>::kBytes
                                                                   : SB0;
  constexpr int SMEM = QBYTES + SBYTES + Sel::kBytes;
  static_assert(MW % G == 0 && ((MWP * 16) & (MWP * 16 - 1)) == 0, "pass shape");
  static_assert(SEL != 0 || RP % (4 * (NT / BN)) == 0, "slice shape");
  static_assert(SEL != 0 || WV * 4 * (KS <= 5 ? 1 : (KS <= 8 ? 2 : 4)) * BN * 4 <= SBYTES,
                "group values of the register epilogue fit in the score tile");
  __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];
  unsigned char* qslots = smem;
  float* S = reinterpret_cast<float*>(smem + QBYTES);
  unsigned char* scratch = smem + QBYTES + SBYTES;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const long long L = logical_block();
  const int qb = (int)(L % a.n_qblocks);
  const long long chunk = L / a.n_qblocks;
  const int q0 = qb * BN;
  const int q_lim = min(BN, a.nq - q0);
  const long long row_begin = chunk * a.rows_per_chunk;
  const long long row_end = min(row_begin + a.rows_per_chunk, a.n_rows);
  const int d = a.d;
  const int nk = d / KC;                                            // k-steps per tile
  const int n_tiles = (int)((row_end - row_begin + TR - 1) / TR);   // 0 for an empty chunk
  const int n_st = n_tiles * nk;
  const T* X = static_cast<const T*>(a.X);
  const T* Qb = static_cast<const T*>(a.Q) + (long long)q0 * d;
  const int kl = (lane >> 4) * 8;  // this lane's 8 dimensions inside a k-step

  Sel sel;
  sel.init();
  if constexpr (kFilt) {
    if (tid < BN) SelFilter<BN>::staged(scratch)[tid] = 0;
    // no barrier needed here: the first tile's epilogue follows several barriers
  }
  float dmn[NW], dmx[NW];  // score dump: this lane's minimum and maximum per query slot
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    dmn[ni] = __builtin_inff();
    dmx[ni] = -__builtin_inff();
  }
  float th[NW];  // filtered mode: thresholds of this lane's query slots
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    const int q = q0 + ni * 16 + (lane & 15);
    th[ni] = q >= a.nq ? __builtin_inff() : (a.th ? a.th[(long long)q * a.th_stride] : kNegInf);
  }
  if (n_st > 0) {
    // Query piece p = tid + NT j: row r = p / 16, 16-byte column c = p % 16 of the
    // super-step, stored at column c ^ (r % 16) of the row.  Any 16 consecutive lanes then
    // touch 256 distinct bytes modulo 256 (all 64 banks), for the row-wise writes and for
    // the fragment reads (16 rows, one column) alike.
    // Loads go through buffer resources: query rows past the batch and tile rows past the
    // index read as zeros (their scores are never selected), with no clamping per lane.
    int qoff[QPT], qdst[QPT];
#pragma unroll
    for (int j = 0; j < QPT; ++j) {
      const int p = tid + NT * j;
      const int r = p / 16, c = p % 16;
      qoff[j] = (r * d + c * 8) * 2;
      qdst[j] = r * 256 + ((c ^ (r & 15)) * 16);
    }
    int xoff[MW];  // byte offset of this lane's 16 bytes of subtile mi inside a k-step of a tile
#pragma unroll
    for (int mi = 0; mi < MW; ++mi) xoff[mi] = ((w * MW * 16 + (lane & 15) + mi * 16) * d + kl) * 2;
    const long long x_end = a.n_rows * (long long)d;  // elements of the index
    const long long q_end = (long long)(a.nq - q0) * d;
    const int fbase = (lane & 15) * 256;  // this lane's query row in fragment ni is 16 ni + lane % 16
    const int fsw = lane & 15;           // n % 16 is lane % 16 for every fragment row
    const int fcol = lane >> 4;          // column of k-step 0; k-step j adds 4 j

    V xr[RS][MW];
    u32x4 qr[QPT];
    V fb[NW];
    f32x4 acc[MW][NW];
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int ni = 0; ni < NW; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

    // One buffer resource per operand: rows from the chunk's first row to the end of the
    // index (the planner keeps a chunk under 2^30 bytes, so 32-bit offsets reach past its
    // end), and the block's queries.  Scalar cursors: x_ahead = byte offset of the next
    // k-step to load (k-step c_ahead of its tile), uq = the next query super-step (the
    // queries repeat for every tile).  Past the chunk the loads read other rows, or zeros
    // past the index, and are never selected from.
    const long long e_chunk = row_begin * d;
    const __amdgpu_buffer_rsrc_t r_x = buffer_rsrc(X + e_chunk, (x_end - e_chunk) * 2);
    const __amdgpu_buffer_rsrc_t r_q = buffer_rsrc(Qb, q_end * 2);
    int x_ahead = 0, c_ahead = 0, uq = 0;
    const int nq4 = nk / 4;
    const int tile_skip = (TR - 1) * d * 2;  // from past a tile's last k-step to the next tile
#define OPRAG_ROWS(SLOT)                                                                 \
  {                                                                                      \
    _Pragma("unroll") for (int mi = 0; mi < MW; ++mi) xr[SLOT][mi] =                     \
        __builtin_bit_cast(V, buffer_load16(r_x, xoff[mi] + x_ahead));                   \
    const bool wrap_ = ++c_ahead == nk;                                                  \
    c_ahead = wrap_ ? 0 : c_ahead;                                                       \
    x_ahead += KC * 2 + (wrap_ ? tile_skip : 0);                                         \
  }
#define OPRAG_QUERIES()                                                                  \
  {                                                                                      \
    _Pragma("unroll") for (int j = 0; j < QPT; ++j) qr[j] =                              \
        buffer_load16(r_q, qoff[j] + uq * (SK * 2));                                     \
    uq = uq + 1 == nq4 ? 0 : uq + 1;                                                     \
  }
#define OPRAG_BFRAG(QS, J)                                                               \
  _Pragma("unroll") for (int ni = 0; ni < NW; ++ni) fb[ni] =                             \
      *reinterpret_cast<const V*>((QS) + fbase + ni * 4096 + (((4 * (J) + fcol) ^ fsw) * 16));
// One k-step: B operand ni of the next k-step (same slot) is read as soon as the MFMAs of
// this k-step are done with fb[ni], so a single set of B registers stays one k-step ahead.
#define OPRAG_KSTEP(U, J, QS)                                                            \
  {                                                                                      \
    OPRAG_ROWS(((U) + PX) % RS)                                                          \
    _Pragma("unroll") for (int ni = 0; ni < NW; ++ni) {                                  \
      _Pragma("unroll") for (int mi = 0; mi < MW; ++mi)                                  \
          acc[mi][ni] = M::run(xr[(U) % RS][mi], fb[ni], acc[mi][ni]);                   \
      if ((J) < 3)                                                                       \
        fb[ni] = *reinterpret_cast<const V*>((QS) + fbase + ni * 4096 +                  \
                                             (((4 * (J) + 4 + fcol) ^ fsw) * 16));       \
    }                                                                                    \
  }
#define OPRAG_SUPER(H)                                                                   \
  {                                                                                      \
    if constexpr (QR > 0) {                                                              \
      unsigned char* qs = qslots + qsi * QSLOT;                                          \
      qsi = qsi + 1 == nq4 ? 0 : qsi + 1;                                                \
      unsigned char* qn = qslots + qsi * QSLOT;                                          \
      OPRAG_KSTEP(4 * (H) + 0, 0, qs)                                                    \
      OPRAG_KSTEP(4 * (H) + 1, 1, qs)                                                    \
      OPRAG_KSTEP(4 * (H) + 2, 2, qs)                                                    \
      OPRAG_KSTEP(4 * (H) + 3, 3, qs)                                                    \
      /* the previous tile's stage flushes are done (filtered mode: if it looked at the  \
         stage) */                                                                       \
      if ((H) == 0 && s0 == t * nk &&                                                    \
          (!kFilt || SEL == 4 || (t > 0 && ((t - 1) & (kFiltCheck - 1)) == kFiltCheck - 1))) \
        lds_barrier();                                                                   \
      OPRAG_BFRAG(qn, 0)                                                                 \
    } else {                                                                             \
      const int sup = s0 / 4 + (H);                                                      \
      unsigned char* qs = qslots + (sup & 1) * QSLOT;                                    \
      unsigned char* qn = qslots + ((sup + 1) & 1) * QSLOT;                              \
      OPRAG_KSTEP(4 * (H) + 0, 0, qs)                                                    \
      OPRAG_KSTEP(4 * (H) + 1, 1, qs)                                                    \
      OPRAG_KSTEP(4 * (H) + 2, 2, qs)                                                    \
      OPRAG_KSTEP(4 * (H) + 3, 3, qs)                                                    \
      _Pragma("unroll") for (int j = 0; j < QPT; ++j)                                    \
          *reinterpret_cast<u32x4*>(qn + qdst[j]) = qr[j];                               \
      OPRAG_QUERIES()                                                                    \
      lds_barrier();                                                                     \
      OPRAG_BFRAG(qn, 0)                                                                 \
    }                                                                                    \
  }

    int qsi = 0;  // resident queries: slot of the current super-step
    if constexpr (QR > 0) {
      // prologue: every super-step of the queries into its own slot (QB super-steps' loads in
      // flight at once), then rows of k-steps 0 .. PX-1
      constexpr int QB = QPT >= 8 ? 1 : 8 / QPT;
      if (SEL == 0 && QB > 1 && nq4 <= QB) {
        // one batch (the small-batch lists kernel): every super-step's queries, then the rows
        // of k-steps 0 .. PX-1, then the queries to their slots, so the wait for the queries
        // leaves the rows in flight
        u32x4 qb[QB][QPT];
#pragma unroll
        for (int u = 0; u < QB; ++u)
#pragma unroll
          for (int j = 0; j < QPT; ++j) qb[u][j] = buffer_load16(r_q, qoff[j] + min(u, nq4 - 1) * (SK * 2));
        __builtin_amdgcn_sched_barrier(0);  // keep the queries ahead of the rows in the load order
#pragma unroll
        for (int u = 0; u < PX; ++u) OPRAG_ROWS(u)
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < QB; ++u)
#pragma unroll
          for (int j = 0; j < QPT; ++j)
            if (u < nq4) *reinterpret_cast<u32x4*>(qslots + u * QSLOT + qdst[j]) = qb[u][j];
      } else {
        for (int u0 = 0; u0 < nq4; u0 += QB) {
          u32x4 qb[QB][QPT];
#pragma unroll
          for (int u = 0; u < QB; ++u)
#pragma unroll
            for (int j = 0; j < QPT; ++j)
              if (QB == 1 || u0 + u < nq4) qb[u][j] = buffer_load16(r_q, qoff[j] + (u0 + u) * (SK * 2));
#pragma unroll
          for (int u = 0; u < QB; ++u)
#pragma unroll
            for (int j = 0; j < QPT; ++j)
              if (QB == 1 || u0 + u < nq4) *reinterpret_cast<u32x4*>(qslots + (u0 + u) * QSLOT + qdst[j]) = qb[u][j];
        }
#pragma unroll
        for (int u = 0; u < PX; ++u) OPRAG_ROWS(u)
      }
    } else {
      // prologue: queries of super-step 0 first (their wait then leaves the row loads in
      // flight), rows of k-steps 0 .. PX-1, queries of super-step 0 to slot 0, queries of
      // super-step 1
      OPRAG_QUERIES()
#pragma unroll
      for (int u = 0; u < PX; ++u) OPRAG_ROWS(u)
#pragma unroll
      for (int j = 0; j < QPT; ++j) *reinterpret_cast<u32x4*>(qslots + qdst[j]) = qr[j];
      OPRAG_QUERIES()
    }
    lds_barrier();
    OPRAG_BFRAG(qslots, 0)

    // Tiles one after another; BODY divides the k-steps of a tile, so ring slots are
    // literal, and the ring runs across tile boundaries (the next tile's first rows are in
    // flight during a tile's selection).
    for (int t = 0; t < n_tiles; ++t) {
#pragma unroll
      for (int mi = 0; mi < MW; ++mi)
#pragma unroll
        for (int ni = 0; ni < NW; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int s0 = t * nk; s0 < (t + 1) * nk; s0 += BODY) {
        OPRAG_SUPER(0)
        if constexpr (BODY >= 8) OPRAG_SUPER(1)
        if constexpr (BODY == 16) {
          OPRAG_SUPER(2)
          OPRAG_SUPER(3)
        }
      }
      // ---- selection for the tile: registers first, else G passes through LDS
      const long long tile0 = row_begin + (long long)t * TR;
      bool refresh = false;  // the group path ran: thresholds and lists of the fast path to restore
      bool done = false;
      if constexpr (SEL == 3) {
        dump_tile<BN, MW, WV>(acc, tile0, row_end, q0, q_lim, a, dmn, dmx);
        done = true;
      } else if constexpr (kFilt) {
        if (a.th == nullptr)  // launch-uniform
          filt_all_tile<BN, MW, WV>(acc, tile0, row_end, q0, q_lim, a);
        else
          filt_tile<SEL == 4, BN, MW, WV>(acc, th, scratch, tile0, row_end, q0, q_lim, t == n_tiles - 1,
                                          SEL == 4 || (t & (kFiltCheck - 1)) == kFiltCheck - 1, a);
        done = true;
      } else if constexpr (SEL == 0) {
        // A chunk's first tile fills the lists through the group path; the tiles after it
        // test against the running thresholds, and take the group path only when a query has
        // too many hits.  (The 128-query k <= 5 kernel keeps the block path for every tile.)
        if constexpr (!kBlk)
          if (t > 0) done = thr_epilogue<BN, MW, WV>(acc, sel, scratch, tile0, row_end, q_lim, a.k);
        if (!done) {
          if constexpr (kBlk)
            done = blk_epilogue<BN, MW, WV>(acc, sel, reinterpret_cast<unsigned char*>(S), scratch, tile0, row_end,
                                            q_lim, a.k, t == 0);
          else if constexpr (kRank)
            done = rank_epilogue<BN, MW, KS, WV>(acc, sel, reinterpret_cast<unsigned char*>(S), scratch, tile0,
                                                 row_end, q_lim, a.k);
          else if (kTileRank && t == 0) {
            if constexpr (kTileRank) first_tile_rank<KS, WV>(acc, sel, scratch, tile0, row_end, q_lim, a.k);
            done = true;
          } else
            done = reg_epilogue<BN, MW, KS, WV>(acc, sel, S, scratch, tile0, row_end, q_lim, a.k);
          refresh = true;
        }
      }
      if (!done) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
#pragma unroll
          for (int mi = g * MWP; mi < (g + 1) * MWP; ++mi)
#pragma unroll
            for (int ni = 0; ni < NW; ++ni) {
              const int q = ni * 16 + (lane & 15);
              const int rl = w * MWP * 16 + (mi - g * MWP) * 16 + (lane >> 4) * 4;
              *reinterpret_cast<f32x4*>(S + q * SR + rl) = acc[mi][ni];
            }
          PassRows pr;
          pr.tile0 = tile0;
          pr.blk = MWP * 16;
          pr.blk_stride = MW * 16;
          pr.off = g * MWP * 16;
          int nv = 0;
#pragma unroll
          for (int bb = 0; bb < WV; ++bb) {
            const long long start = tile0 + (long long)bb * MW * 16 + g * MWP * 16;
            nv += (int)max(0ll, min((long long)(MWP * 16), row_end - start));
          }
          pr.nvalid = nv;
          lds_barrier();
          sel.pass(S, SR, RP, pr, q_lim, a.k, scratch);
        }
      }
      if constexpr (SEL == 0 && !kBlk)
        if (refresh) thr_reset(sel, scratch, q_lim, a.k, BN);
    }
#undef OPRAG_SUPER
#undef OPRAG_KSTEP
#undef OPRAG_BFRAG
#undef OPRAG_QUERIES
#undef OPRAG_ROWS
  }
  if constexpr (kFilt) {
    if (a.th == nullptr) {
      if (chunk == 0 && tid < q_lim) a.ccnt[q0 + tid] = (int)a.n_rows;  // every row is a candidate
    }  // else the chunk's last tile flushed its stages
  } else if constexpr (SEL == 3) {
    if (a.dump_mm != nullptr) {  // launch-uniform
      // the four lanes of a query slot in a wave, then the waves through LDS
#pragma unroll
      for (int ni = 0; ni < NW; ++ni) {
        dmn[ni] = fminf(dmn[ni], __shfl_xor(dmn[ni], 16));
        dmx[ni] = fmaxf(dmx[ni], __shfl_xor(dmx[ni], 16));
        dmn[ni] = fminf(dmn[ni], __shfl_xor(dmn[ni], 32));
        dmx[ni] = fmaxf(dmx[ni], __shfl_xor(dmx[ni], 32));
      }
      __syncthreads();  // every wave is done with the query slots, reused here
      float* red = reinterpret_cast<float*>(qslots);  // [WV][BN][2]
      static_assert(WV * BN * 2 * 4 <= QBYTES, "reduction area");
      if (lane < 16) {
#pragma unroll
        for (int ni = 0; ni < NW; ++ni) {
          red[(w * BN + ni * 16 + lane) * 2] = dmn[ni];
          red[(w * BN + ni * 16 + lane) * 2 + 1] = dmx[ni];
        }
      }
      __syncthreads();
      if (tid < q_lim) {
        float mn = __builtin_inff(), mx = -__builtin_inff();
#pragma unroll
        for (int u = 0; u < WV; ++u) {
          mn = fminf(mn, red[(u * BN + tid) * 2]);
          mx = fmaxf(mx, red[(u * BN + tid) * 2 + 1]);
        }
        float* o = a.dump_mm + ((long long)(q0 + tid) * a.n_chunks + chunk) * 2;
        o[0] = mn;
        o[1] = mx;
      }
    }
  } else {
    sel.write(a, q0, chunk);
  }
}

#undef OPRAG_DENSE_KERNEL

#ifdef OPRAG_DENSE_ILP
#define OPRAG_ILP_INSTANCE(DT, NW, MW, RS, G, KS, SEL, WV, QR) \
  template __global__ void dense_mfma_kernel_ilp<DT, NW, MW, RS, G, KS, SEL, WV, QR>(DenseArgs);
OPRAG_ILP_KERNELS(OPRAG_ILP_INSTANCE, kDtypeBF16)
OPRAG_ILP_KERNELS(OPRAG_ILP_INSTANCE, kDtypeF16)
#undef OPRAG_ILP_INSTANCE

}  // namespace oprag
#else  // the rest of the library's dense search: other kernels, the kernel table, planning

// ------------------------------------------------------------------------------------
// fp32 VALU kernel: tile of 64 rows x 32 queries, 32 dimensions per stage.
// ------------------------------------------------------------------------------------
template <int KS, int SEL>
__global__ __launch_bounds__(kThreads) void dense_f32_kernel(DenseArgs a) {
  constexpr int BN = 32, TR = 64, KC = 32, SR = TR + 4;
  using Sel = typename SelOf<BN, KS, SEL, kThreads>::type;
  constexpr int XB = TR * (KC + 1) * 4, QB = BN * (KC + 1) * 4;
  constexpr int SB = BN * SR * 4;
  constexpr int A1 = XB + QB;
  constexpr int A2 = SB + Sel::kBytes;
  constexpr int SMEM = A1 > A2 ? A1 : A2;
  __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];
  float* Xs = reinterpret_cast<float*>(smem);
  float* Qs = reinterpret_cast<float*>(smem + XB);

  const int tid = threadIdx.x;
  const long long L = logical_block();
  const int qb = (int)(L % a.n_qblocks);
  const long long chunk = L / a.n_qblocks;
  const int q0 = qb * BN;
  const int q_lim = min(BN, a.nq - q0);
  const long long row_begin = chunk * a.rows_per_chunk;
  const long long row_end = min(row_begin + a.rows_per_chunk, a.n_rows);
  const int d = a.d;
  const float* X = static_cast<const float*>(a.X);
  const float* Q = static_cast<const float*>(a.Q);
  const int qq = tid % BN, rg = tid / BN;  // query, group of 8 rows

  Sel sel;
  sel.init();

  // Each thread stages two 16-byte row pieces and one query piece per stage; the next
  // stage's pieces are loaded while the current one is multiplied.
  const int pc = tid % (KC / 4);                // 16-byte column of the stage
  const int pr0 = tid / (KC / 4);               // row of piece 0 (rows pr0 and pr0 + 32)
  const int qrow = min(q0 + pr0, a.nq - 1);
  float4 xa, xb, qa;
  auto fetch = [&](long long tile, int kc) __attribute__((always_inline)) {
    const bool in = kc + pc * 4 < d;
    const long long r0 = min(tile + pr0, a.n_rows - 1), r1 = min(tile + pr0 + 32, a.n_rows - 1);
    xa = in ? *reinterpret_cast<const float4*>(X + r0 * d + kc + pc * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
    xb = in ? *reinterpret_cast<const float4*>(X + r1 * d + kc + pc * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
    qa = in ? *reinterpret_cast<const float4*>(Q + (long long)qrow * d + kc + pc * 4)
            : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  if (row_begin < row_end) fetch(row_begin, 0);
  for (long long tile0 = row_begin; tile0 < row_end; tile0 += TR) {
    float acc[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) acc[r] = 0.f;
    for (int kc = 0; kc < d; kc += KC) {
      __syncthreads();
      float* xd0 = Xs + pr0 * (KC + 1) + pc * 4;
      float* xd1 = Xs + (pr0 + 32) * (KC + 1) + pc * 4;
      float* qd = Qs + pr0 * (KC + 1) + pc * 4;
      xd0[0] = xa.x, xd0[1] = xa.y, xd0[2] = xa.z, xd0[3] = xa.w;
      xd1[0] = xb.x, xd1[1] = xb.y, xd1[2] = xb.z, xd1[3] = xb.w;
      qd[0] = qa.x, qd[1] = qa.y, qd[2] = qa.z, qd[3] = qa.w;
      if (kc + KC < d)
        fetch(tile0, kc + KC);
      else if (tile0 + TR < row_end)
        fetch(tile0 + TR, 0);
      __syncthreads();
#pragma unroll 4
      for (int c = 0; c < KC; ++c) {
        const float qv = Qs[qq * (KC + 1) + c];
#pragma unroll
        for (int r = 0; r < 8; ++r) acc[r] = __builtin_fmaf(Xs[(rg * 8 + r) * (KC + 1) + c], qv, acc[r]);
      }
    }
    __syncthreads();
    float* S = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int r = 0; r < 8; ++r) S[qq * SR + rg * 8 + r] = acc[r];
    PassRows pr;
    pr.tile0 = tile0;
    pr.blk = TR;
    pr.blk_stride = TR;
    pr.off = 0;
    pr.nvalid = (int)min((long long)TR, row_end - tile0);
    __syncthreads();
    sel.pass(S, SR, TR, pr, q_lim, a.k, smem + SB);
    __syncthreads();
  }
  sel.write(a, q0, chunk);
}

// ------------------------------------------------------------------------------------
// Filtered mode, selection: exact top-k (sorted) of a query's candidate keys.  One workgroup
// of NT threads per query: 1,024 when one round of workgroups covers the batch (the query's
// latency counts), 256 for larger batches (more queries per CU at once).  Keys are unique
// composites (row ids are), so exactly min(k, n) keys qualify.  Buffers of up to 4,096 keys
// are read once (all loads in flight) and kept in registers.  The 256 groups of NT / 256
// adjacent threads take their largest key, and tau = the need-th largest of these maxima
// bounds the need-th best key from below (every maximum is a key of its own); the keys >= tau
// are ranked exactly.  Too many of them, or larger buffers, take a most-significant-digit
// radix select (8-bit digits, stopping as soon as a whole bucket is needed).
// ------------------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(NT) void select_topk_kernel(const unsigned long long* __restrict__ cbuf,
                                                         int* __restrict__ ccnt, long long cap, int k,
                                                         float* out_scores, long long* out_ids, int* overflow,
                                                         const int* gate, int threshold_only) {
  constexpr int kCand = 1024;  // candidates the threshold path ranks directly
  constexpr int kRegKeys = 4096 / NT;
  constexpr int GS = NT / 256;        // threads per group
  constexpr int GB = 256 / GS;        // group maxima each thread of a group counts over
  constexpr int GST = GB + 2;         // block stride: the GS blocks start in different banks
  static_assert(NT == 256 || NT == 1024, "workgroup size");
  __shared__ u64 cand[kCand];
  __shared__ __attribute__((aligned(16))) u64 gmax[GS * GST];
  __shared__ u64 s_tau;
  __shared__ int s_nc;
  __shared__ unsigned int hist[256];
  __shared__ int wtot[NT / 64];
  __shared__ u64 sel[kMaxK];
  __shared__ u64 s_prefix, s_mask;
  __shared__ int s_need, s_done, s_ns;
  if (gate != nullptr && *gate == 0) return;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int q = blockIdx.x;
  const int cnt = ccnt[q];
  if (t == 0 && cnt > cap && overflow != nullptr) atomicAdd(overflow, 1);
  const int n = (int)min((long long)cnt, cap);
  const u64* src = cbuf + (long long)q * cap;
  if (t == 0) {
    s_prefix = 0ull;
    s_mask = 0ull;
    s_need = min(k, n);
    s_done = s_need == 0;
    s_ns = 0;
    s_tau = 0ull;
  }
  __syncthreads();
  if (t == 0) ccnt[q] = 0;  // every thread has read it: the next pass starts from zero
  const int need = min(k, n);
  const bool in_reg = n <= kRegKeys * NT;  // workgroup-uniform
  // Register keys: thread t holds keys ib + NT u, where ib puts the first 256 keys in 256
  // different groups, so at least min(n, 256) >= need groups are nonempty.
  const int ib = t / GS + 256 * (t % GS);
  u64 kv[kRegKeys];
  if (in_reg) {
#pragma unroll
    for (int u = 0; u < kRegKeys; ++u) {
      const int i = ib + u * NT;
      kv[u] = i < n ? src[i] : 0ull;
    }
  }
  // keys of this thread beyond the registers, eight loads in flight per step
  auto scan_global = [&](auto&& f) __attribute__((always_inline)) {
    for (int i0 = t; i0 < n; i0 += 8 * NT) {
      u64 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = i0 + u * NT < n ? src[i0 + u * NT] : 0ull;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (i0 + u * NT < n) f(v[u]);
    }
  };
  if (need > 0) {
    u64 m = 0ull;
    if (in_reg) {
#pragma unroll
      for (int u = 0; u < kRegKeys; ++u) m = umax64(m, kv[u]);
    } else {
      scan_global([&](u64 x) { m = umax64(m, x); });
    }
#pragma unroll
    for (int o = 1; o < GS; o <<= 1) m = umax64(m, shfl_xor64(m, o));
    const int grp = t / GS, sub = t % GS;
    if (sub == 0) gmax[(grp / GB) * GST + grp % GB] = m;
    __syncthreads();
    // each of the group's threads counts the larger maxima in its share of the list
    int gt = 0;
    const u64* blk = gmax + sub * GST;
#pragma unroll 16
    for (int u = 0; u < GB; ++u) gt += blk[u] > m ? 1 : 0;
#pragma unroll
    for (int o = 1; o < GS; o <<= 1) gt += __shfl_xor(gt, o);
    // nonzero maxima are unique, and at least need groups hold keys
    if (sub == 0 && m != 0ull && gt == need - 1) s_tau = m;
    __syncthreads();
    const u64 tau = s_tau;
    if (threshold_only) {
      // An earlier level only hands its k-th score on as the next threshold, and tau is a
      // valid one: at least k keys reach it (k <= n here, else the next level takes all rows).
      if (t == 0) out_scores[(long long)q * k + (k - 1)] = need == k ? comp_score(tau) : kNegInf;
      return;
    }
    int c = 0;
    if (in_reg) {
#pragma unroll
      for (int u = 0; u < kRegKeys; ++u) c += (ib + u * NT < n && kv[u] >= tau) ? 1 : 0;
    } else {
      scan_global([&](u64 x) { c += x >= tau ? 1 : 0; });
    }
    // exclusive scan of c over the workgroup
    int x = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) wtot[w] = x;
    __syncthreads();
    int pos = x - c;
    for (int i = 0; i < w; ++i) pos += wtot[i];
    if (t == NT - 1) s_nc = pos + c;
    __syncthreads();
    const int nc = s_nc;
    if (nc <= kCand) {  // workgroup-uniform
      if (in_reg) {
#pragma unroll
        for (int u = 0; u < kRegKeys; ++u)
          if (ib + u * NT < n && kv[u] >= tau) cand[pos++] = kv[u];
      } else {
        scan_global([&](u64 x) {
          if (x >= tau) cand[pos++] = x;
        });
      }
      __syncthreads();
      // rank = number of larger keys; L adjacent lanes share a candidate, each comparing
      // every L-th entry
      int lg = 0;
      while (lg < 4 && (nc << (lg + 1)) <= NT) ++lg;
      const int L = 1 << lg, jc = t >> lg, p = t & (L - 1);
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
      if (jc < nc && p == 0 && r < need) {
        out_ids[(long long)q * k + r] = (long long)comp_row(me);
        out_scores[(long long)q * k + r] = comp_score(me);
      }
      for (int r2 = need + t; r2 < k; r2 += NT) {
        out_ids[(long long)q * k + r2] = -1ll;
        out_scores[(long long)q * k + r2] = kNegInf;
      }
      return;
    }
  }
  for (int shift = 56; shift >= 0; shift -= 8) {
    if (s_done) break;  // block-uniform
    const u64 prefix = s_prefix, mask = s_mask;
    const int need_d = s_need;
    if (t < 256) hist[t] = 0u;
    __syncthreads();
    auto count = [&](u64 key) __attribute__((always_inline)) {
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    };
    if (in_reg) {
#pragma unroll
      for (int u = 0; u < kRegKeys; ++u)
        if (ib + u * NT < n) count(kv[u]);
    } else {
      scan_global(count);
    }
    __syncthreads();
    // threads 0 .. 255 (waves 0 .. 3): thread t holds digit 255 - t; an inclusive scan over t
    // counts the keys whose digit is >= 255 - t within the prefix bucket
    int hd = 0, x = 0;
    if (t < 256) {
      hd = (int)hist[255 - t];
      x = hd;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
      }
      if (lane == 63) wtot[w] = x;
    }
    __syncthreads();
    if (t < 256) {
      int before = 0;
      for (int i = 0; i < w; ++i) before += wtot[i];
      const int incl = before + x;          // keys with digit >= 255 - t
      const int above = incl - hd;          // keys with digit > 255 - t
      if (above < need_d && incl >= need_d) {  // exactly one thread: the digit of the k-th key
        const int dgt = 255 - t;
        s_prefix = prefix | ((u64)dgt << shift);
        s_mask = mask | (255ull << shift);
        s_need = need_d - above;
        s_done = (hd == need_d - above) ? 1 : 0;  // the whole bucket is needed: stop here
      }
    }
    __syncthreads();
  }
  const u64 prefix = s_prefix, mask = s_mask;
  auto gather = [&](u64 key) __attribute__((always_inline)) {
    if ((key & mask) >= prefix) {
      const int slot = atomicAdd(&s_ns, 1);
      if (slot < kMaxK) sel[slot] = key;
    }
  };
  if (in_reg) {
#pragma unroll
    for (int u = 0; u < kRegKeys; ++u)
      if (ib + u * NT < n) gather(kv[u]);
  } else {
    scan_global(gather);
  }
  __syncthreads();
  const int ns = min(s_ns, k);  // == min(k, n)
  if (t < ns) {
    const u64 key = sel[t];
    int rank = 0;
    for (int j = 0; j < ns; ++j) rank += sel[j] > key ? 1 : 0;
    out_ids[(long long)q * k + rank] = (long long)comp_row(key);
    out_scores[(long long)q * k + rank] = comp_score(key);
  }
  for (int r = ns + t; r < k; r += NT) {
    out_ids[(long long)q * k + r] = -1ll;
    out_scores[(long long)q * k + r] = kNegInf;
  }
}

// Weighted fusion (Section 4.4): per query, the dense and lexical scores of every chunk,
// min-max normalised over all chunks (a constant row normalises to 0), weighted and summed in
// fp64 and rounded to fp32.  Lexical scores past n_lex chunks are 0.  One workgroup of 1,024
// threads per query; eight chunks per thread and step, their loads issued before use.
//   pass 1: the minima and maxima of both rows, from the dumps' per-chunk / per-range
//           partials (and 0 for the lexical row when chunks past n_lex exist);
//   pass 2: every chunk's fused composite; tau = the need-th largest of the maxima of the 128
//           eight-thread groups (need = min(k, n) <= 128) bounds the need-th best composite
//           from below;
//   pass 3: the same composites again, and those >= tau go to cbuf[q] (in any order) with
//           their count in ccnt[q], for the exact selection.
// Pass 2 keeps the score keys of the first kFuseLds chunks in LDS for pass 3 and the rest are
// computed again; every operation is rounded explicitly, so both ways give the same composites.
constexpr int kFuseThreads = 1024, kFuseGroups = kFuseThreads / 8, kFuseLds = 32768;
static_assert(kFuseLds % (8 * kFuseThreads) == 0, "whole steps come from LDS");
static_assert(kMaxK <= kFuseGroups, "tau needs k group maxima");
__device__ __forceinline__ u64 fused_composite(double sd, double sl, double mnd, double mnl, float x, float y,
                                               long long i) {
  return composite(fused_value(sd, sl, mnd, mnl, x, y), (uint32_t)i);
}
__global__ __launch_bounds__(kFuseThreads) void weighted_fuse_kernel(const float* __restrict__ D,
                                                                 const float* __restrict__ B, long long ld,
                                                                 long long n, long long n_lex,
                                                                 const float* __restrict__ mm_d, int pd,
                                                                 const float* __restrict__ mm_l, int pl, double wd,
                                                                 double wl, int k, unsigned long long* cbuf, int* ccnt) {
  __shared__ float red[4][kFuseThreads / 64];
  __shared__ uint32_t skey[kFuseLds];
  __shared__ u64 gmax[kFuseGroups];
  __shared__ u64 s_tau;
  __shared__ int s_cnt;
  const long long q = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const float* d = D + q * ld;
  const float* b = B + q * ld;
  float mnd = __builtin_inff(), mxd = -__builtin_inff(), mnl = __builtin_inff(), mxl = -__builtin_inff();
  for (int i = t; i < pd; i += kFuseThreads) {
    mnd = fminf(mnd, mm_d[(q * pd + i) * 2]);
    mxd = fmaxf(mxd, mm_d[(q * pd + i) * 2 + 1]);
  }
  for (int i = t; i < pl; i += kFuseThreads) {
    mnl = fminf(mnl, mm_l[(q * pl + i) * 2]);
    mxl = fmaxf(mxl, mm_l[(q * pl + i) * 2 + 1]);
  }
  if (n_lex < n) {  // chunks past the sparse corpus score 0 lexically
    mnl = fminf(mnl, 0.f);
    mxl = fmaxf(mxl, 0.f);
  }
  for (int o = 32; o > 0; o >>= 1) {
    mnd = fminf(mnd, __shfl_xor(mnd, o));
    mxd = fmaxf(mxd, __shfl_xor(mxd, o));
    mnl = fminf(mnl, __shfl_xor(mnl, o));
    mxl = fmaxf(mxl, __shfl_xor(mxl, o));
  }
  if (lane == 0) {
    red[0][w] = mnd;
    red[1][w] = mxd;
    red[2][w] = mnl;
    red[3][w] = mxl;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kFuseThreads / 64; ++u) {
    mnd = fminf(mnd, red[0][u]);
    mxd = fmaxf(mxd, red[1][u]);
    mnl = fminf(mnl, red[2][u]);
    mxl = fmaxf(mxl, red[3][u]);
  }
  const double sd = mxd > mnd ? wd / ((double)mxd - (double)mnd) : 0.0;
  const double sl = mxl > mnl ? wl / ((double)mxl - (double)mnl) : 0.0;
  const double mnd64 = mnd, mnl64 = mnl;
  // pass 2: this thread's largest composite, then its group's
  u64 m = 0ull;
  for (long long i0 = t; i0 < n; i0 += 8 * kFuseThreads) {
    float x[8], y[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const long long i = i0 + (long long)u * kFuseThreads;
      x[u] = i < n ? d[i] : 0.f;
      y[u] = i < n_lex ? b[i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const long long i = i0 + (long long)u * kFuseThreads;
      if (i < n) {
        const u64 c = fused_composite(sd, sl, mnd64, mnl64, x[u], y[u], i);
        m = umax64(m, c);
        if (i < kFuseLds) skey[i] = comp_key(c);
      }
    }
  }
#pragma unroll
  for (int o = 1; o < 8; o <<= 1) m = umax64(m, __shfl_xor(m, o));
  if ((t & 7) == 0) gmax[t >> 3] = m;
  if (t == 0) {
    s_tau = 0ull;
    s_cnt = 0;
  }
  __syncthreads();
  // Nonzero group maxima are distinct composites; when fewer than need of them exist, tau
  // stays 0 and every chunk is a candidate.
  const int need = (int)min((long long)k, n);
  if (t < kFuseGroups && need > 0) {
    const u64 g = gmax[t];
    int gt = 0;
#pragma unroll 8
    for (int u = 0; u < kFuseGroups; ++u) gt += gmax[u] > g ? 1 : 0;
    if (g != 0ull && gt == need - 1) s_tau = g;
  }
  __syncthreads();
  const u64 tau = s_tau;
  // pass 3: compact the composites >= tau, one LDS reservation per wave and step
  unsigned long long* dst = cbuf + q * n;
  for (long long i0 = t; i0 < n; i0 += 8 * kFuseThreads) {
    float x[8], y[8];
    const bool from_lds = i0 + 7ll * kFuseThreads < kFuseLds;  // uniform: whole steps
    if (!from_lds) {
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const long long i = i0 + (long long)u * kFuseThreads;
        x[u] = i < n ? d[i] : 0.f;
        y[u] = i < n_lex ? b[i] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const long long i = i0 + (long long)u * kFuseThreads;
      u64 c = 0ull;
      if (i < n)
        c = from_lds ? ((u64)skey[i] << 32) | (u64)(uint32_t)(~(uint32_t)i)
                     : fused_composite(sd, sl, mnd64, mnl64, x[u], y[u], i);
      const bool take = i < n && c >= tau;
      const u64 bal = __ballot(take);
      if (bal != 0ull) {
        int base = 0;
        if (lane == __ffsll((long long)bal) - 1) base = atomicAdd(&s_cnt, __popcll(bal));
        base = __shfl(base, __ffsll((long long)bal) - 1);
        if (take) dst[base + __popcll(bal & ((1ull << lane) - 1ull))] = c;
      }
    }
  }
  __syncthreads();
  if (t == 0) ccnt[q] = s_cnt;
}

// Clears the filtered-mode counters (a kernel, not a memset: safe inside captured graphs).
__global__ void clear_ints_kernel(int* p, long long n, const int* gate) {
  if (gate != nullptr && *gate == 0) return;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x)
    p[i] = 0;
}

// ------------------------------------------------------------------------------------
// Merge of the per-chunk lists (k <= 16), one wave per query.  The query's n = n_chunks * k
// composites (unique, larger is better, 0 = empty slot) are read in lane-strided order.  The
// k-th largest of the 64 lane maxima is a lower bound tau of the k-th best composite (the k
// lanes from the top each hold a composite at least that large), so the composites >= tau
// are the only candidates; they are compacted into LDS and every candidate's rank is the
// number of candidates larger than it.  With more than 64 candidates the wave instead extracts the k
// best one by one (k rounds of a lane-local and a wave-wide maximum).
// ------------------------------------------------------------------------------------
__device__ __forceinline__ u64 wave_max64(u64 x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = umax64(x, shfl_xor64(x, o));
  return x;
}

// PB: composites per lane per batch, all loaded before any is used; a query whose lists fit one
// batch (64 PB composites) is read once and kept in registers for both passes.
template <int PB>
__global__ __launch_bounds__(kThreads) void merge_lists_kernel(const u64* __restrict__ partial, int n_chunks, int nq,
                                                               int k, float* out_scores, long long* out_ids) {
  __shared__ u64 cand[kWaves][64];
  __shared__ u64 s_tau[kWaves];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const long long q = (long long)blockIdx.x * kWaves + w;
  if (q >= nq) return;  // whole waves; nothing below synchronises the workgroup
  const long long n = (long long)n_chunks * k;
  const u64* src = partial + q * n;
  float* osc = out_scores + q * k;
  long long* oid = out_ids + q * k;
  u64 kb[PB];
  // Row r of 64 composites goes to the lanes rotated by r: the lists are sorted and, when 64 is
  // a multiple of k, an unrotated lane would see the same list position in every row (lanes of
  // the first positions then hold every large maximum, and with k = 16 hundreds of composites
  // reached tau); rotated, each lane's maximum mixes positions and about k composites reach it.
  auto load_batch = [&](long long base) {
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const long long r = (base >> 6) + u;  // base is a multiple of 64
      const long long j = r * 64 + ((lane - (int)(r & 63)) & 63);
      kb[u] = j < n ? src[j] : 0ull;
    }
  };

  u64 m = 0;
  for (long long base = 0; base < n; base += 64 * PB) {
    load_batch(base);
#pragma unroll
    for (int u = 0; u < PB; ++u) m = umax64(m, kb[u]);
  }
  // tau = the lane maximum of rank k - 1 (ranks from LDS broadcast reads; the maxima are
  // unique apart from empty lanes), or 0 when fewer than k lanes hold a composite
  cand[w][lane] = m;
  if (lane == 0) s_tau[w] = 0ull;
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  {
    int rank = 0;
#pragma unroll 8
    for (int u = 0; u < 64; ++u) rank += cand[w][u] > m ? 1 : 0;
    if (rank == k - 1) s_tau[w] = m;
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  const u64 tau = s_tau[w];
  const u64 below = (1ull << lane) - 1ull;
  int c = 0;  // candidates so far (wave-uniform)
  for (long long base = 0; base < n; base += 64 * PB) {
    if (n > 64 * PB) load_batch(base);  // a single batch is still in registers
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const bool take = kb[u] != 0ull && kb[u] >= tau;
      const u64 bal = __ballot(take);
      if (take) {
        const int pos = c + __popcll(bal & below);
        if (pos < 64) cand[w][pos] = kb[u];
      }
      c += __popcll(bal);
    }
  }
  if (c <= 64) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's LDS writes are complete
    const u64 me = lane < c ? cand[w][lane] : 0ull;
    int rank = 0;
    for (int u = 0; u < c; ++u) rank += cand[w][u] > me ? 1 : 0;
    if (lane < c && rank < k) {
      oid[rank] = (long long)comp_row(me);
      osc[rank] = comp_score(me);
    }
    for (int r = c + lane; r < k; r += 64) {
      oid[r] = -1;
      osc[r] = kNegInf;
    }
  } else {
    // at least 64 >= k composites reach tau, so every round finds one
    u64 last = ~0ull;
    for (int r = 0; r < k; ++r) {
      u64 mx = 0;
      for (long long base = 0; base < n; base += 64 * PB) {
        if (n > 64 * PB) load_batch(base);
#pragma unroll
        for (int u = 0; u < PB; ++u)
          if (kb[u] >= tau && kb[u] < last) mx = umax64(mx, kb[u]);
      }
      last = wave_max64(mx);
      if (lane == 0) {
        oid[r] = (long long)comp_row(last);
        osc[r] = comp_score(last);
      }
    }
  }
}

// Long list sets (more than 2,048 composites per query, k <= 16): one workgroup per query.  Wave w
// takes the query's rows of 64 composites [R w / 4, R (w + 1) / 4) (R rows in all), rotated across
// lanes as above, finds their k best exactly by the same steps (lane maxima, tau, the composites
// reaching it ranked in LDS, or k rounds of maxima when more than 64 reach it), and writes them in
// rank order to its list in LDS; the first wave then ranks the four sorted lists against each
// other (lane l holds entry l % 16 of list l / 16).
constexpr int kWgMergeK = 16;
__global__ __launch_bounds__(kThreads) void merge_lists_wg_kernel(const u64* __restrict__ partial, int n_chunks,
                                                                  int nq, int k, float* out_scores,
                                                                  long long* out_ids) {
  constexpr int PB = 16;
  __shared__ u64 cand[kWaves][64];
  __shared__ u64 s_tau[kWaves];
  __shared__ u64 best[kWaves][kWgMergeK];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const long long q = blockIdx.x;  // one query per workgroup: grid = nq
  const long long n = (long long)n_chunks * k;
  const long long rows = (n + 63) / 64;
  const long long r0 = rows * w / kWaves, r1 = rows * (w + 1) / kWaves;
  const u64* src = partial + q * n;
  u64 kb[PB];
  auto load_batch = [&](long long rb) {  // rows rb .. rb + PB - 1 of this wave's range
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const long long r = rb + u;
      const long long j = r * 64 + ((lane - (int)(r & 63)) & 63);
      kb[u] = (r < r1 && j < n) ? src[j] : 0ull;
    }
  };
  u64 m = 0;
  for (long long rb = r0; rb < r1; rb += PB) {
    load_batch(rb);
#pragma unroll
    for (int u = 0; u < PB; ++u) m = umax64(m, kb[u]);
  }
  cand[w][lane] = m;
  if (lane == 0) s_tau[w] = 0ull;
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  {
    int rank = 0;
#pragma unroll 8
    for (int u = 0; u < 64; ++u) rank += cand[w][u] > m ? 1 : 0;
    if (rank == k - 1) s_tau[w] = m;
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  const u64 tau = s_tau[w];
  const u64 below = (1ull << lane) - 1ull;
  const bool one_batch = r1 - r0 <= PB;
  int c = 0;
  for (long long rb = r0; rb < r1; rb += PB) {
    if (!one_batch) load_batch(rb);
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const bool take = kb[u] != 0ull && kb[u] >= tau;
      const u64 bal = __ballot(take);
      if (take) {
        const int pos = c + __popcll(bal & below);
        if (pos < 64) cand[w][pos] = kb[u];
      }
      c += __popcll(bal);
    }
  }
  if (lane < kWgMergeK) best[w][lane] = 0ull;
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  if (c <= 64) {
    const u64 me = lane < c ? cand[w][lane] : 0ull;
    int rank = 0;
    for (int u = 0; u < c; ++u) rank += cand[w][u] > me ? 1 : 0;
    if (lane < c && rank < k) best[w][rank] = me;
  } else {
    // at least 64 >= k composites reach tau, so every round finds one
    u64 last = ~0ull;
    for (int r = 0; r < k; ++r) {
      u64 mx = 0;
      for (long long rb = r0; rb < r1; rb += PB) {
        if (!one_batch) load_batch(rb);
#pragma unroll
        for (int u = 0; u < PB; ++u)
          if (kb[u] >= tau && kb[u] < last) mx = umax64(mx, kb[u]);
      }
      last = wave_max64(mx);
      if (lane == 0) best[w][r] = last;
    }
  }
  __syncthreads();
  if (w == 0) {
    const int li = lane >> 4, pos = lane & 15;
    const u64 x = pos < k ? best[li][pos] : 0ull;
    int rank = pos;
#pragma unroll
    for (int lj = 0; lj < kWaves; ++lj) {
      if (lj == li) continue;
#pragma unroll
      for (int p2 = 0; p2 < kWgMergeK; ++p2) rank += (p2 < k && best[lj][p2] > x) ? 1 : 0;
    }
    float* osc = out_scores + q * k;
    long long* oid = out_ids + q * k;
    if (x != 0ull && rank < k) {
      oid[rank] = (long long)comp_row(x);
      osc[rank] = comp_score(x);
    }
    const int tot = __popcll(__ballot(x != 0ull));
    for (int r = tot + lane; r < k; r += 64) {
      oid[r] = -1;
      osc[r] = kNegInf;
    }
  }
}

// k <= 128: one wave per query keeps a 128-entry queue and merges 64 candidates at a time.
__global__ __launch_bounds__(kThreads) void merge_large_kernel(const unsigned long long* __restrict__ partial,
                                                               int n_chunks, int nq, int k, float* out_scores,
                                                               long long* out_ids, const int* gate) {
  if (gate != nullptr && *gate == 0) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int q = blockIdx.x * kWaves + w;
  if (q >= nq) return;
  const long long n = (long long)n_chunks * k;
  const unsigned long long* src = partial + (long long)q * n;
  u64 q0 = 0ull, q1 = 0ull;
  for (long long base = 0; base < n; base += 256) {
    u64 c[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) c[u] = base + u * 64 + lane < n ? src[base + u * 64 + lane] : 0ull;
#pragma unroll
    for (int u = 0; u < 4; ++u) wave_offer(q0, q1, c[u], queue_at(q0, q1, k - 1), lane);
  }
  const long long o = (long long)q * k;
  if (lane < k) {
    out_ids[o + lane] = q0 ? (long long)comp_row(q0) : -1ll;
    out_scores[o + lane] = q0 ? comp_score(q0) : kNegInf;
  }
  if (lane + 64 < k) {
    out_ids[o + lane + 64] = q1 ? (long long)comp_row(q1) : -1ll;
    out_scores[o + lane + 64] = q1 ? comp_score(q1) : kNegInf;
  }
}

// ------------------------------------------------------------------------------------
// Kernel table and planning.
// ------------------------------------------------------------------------------------
struct KernelInfo {
  void (*fn)(DenseArgs);
  int dtype, bn, tile_rows, ks, sel;
  int chunk_target;  // workgroups per CU the planner aims for (chunks x query blocks / CUs)
  int min_nq, max_nq;
  int ring;     // MFMA kernels: k-steps per loop iteration, which must divide d / 32 (0: none)
  int threads;  // workgroup size
  int qres;     // resident query super-steps (0: streamed); the kernel serves d / 128 <= qres
};

#define MFKQ(DT, NW, MW, RS, G, KS, SEL, OCC, LO, HI, WV, QR)                                              \
  {dense_mfma_kernel<DT, NW, MW, RS, G, KS, SEL, WV, QR>, DT, NW * 16, WV * MW * 16, KS, SEL, OCC, LO, HI, RS, \
   WV * 64, QR}
#define MFKW(DT, NW, MW, RS, G, KS, SEL, OCC, LO, HI, WV) MFKQ(DT, NW, MW, RS, G, KS, SEL, OCC, LO, HI, WV, 0)
#define MFK(DT, NW, MW, RS, G, KS, SEL, OCC, LO, HI) MFKW(DT, NW, MW, RS, G, KS, SEL, OCC, LO, HI, kWaves)
// The same entries for the instances built with the ILP scheduler (OPRAG_ILP_KERNELS).
#define MFKQI(DT, NW, MW, RS, G, KS, SEL, OCC, LO, HI, QR)                                                   \
  {dense_mfma_kernel_ilp<DT, NW, MW, RS, G, KS, SEL, kWaves, QR>, DT, NW * 16, kWaves * MW * 16, KS, SEL, OCC, LO, \
   HI, RS, kWaves * 64, QR}
#define MFKI(DT, NW, MW, RS, G, KS, SEL, OCC, LO, HI) MFKQI(DT, NW, MW, RS, G, KS, SEL, OCC, LO, HI, 0)
// Deep rings first; the 4-deep variants serve dimensions that are not multiples of the ring.
#define MF_KS(DT, NW, MW, RS, G, OCC, LO, HI)                                                   \
  MFK(DT, NW, MW, RS, G, 5, 0, OCC, LO, HI), MFK(DT, NW, MW, RS, G, 8, 0, OCC, LO, HI),          \
      MFK(DT, NW, MW, RS, G, 16, 0, OCC, LO, HI)
#define MF_KSI(DT, NW, MW, RS, G, OCC, LO, HI)                                                  \
  MFKI(DT, NW, MW, RS, G, 5, 0, OCC, LO, HI), MFK(DT, NW, MW, RS, G, 8, 0, OCC, LO, HI),         \
      MFK(DT, NW, MW, RS, G, 16, 0, OCC, LO, HI)
// The single-query-block kernels aim for one workgroup per CU: two 64-row tiles each, so the
// ring streams across a tile boundary and the second tile takes the running-threshold path.
// Their instances for d <= 1,024 keep the block's queries resident in LDS: no query loads
// join the ring's in-order load counter, and one barrier per tile (1.3 to 2 us per call at
// batches 1 and 16).
// The 128-query list kernels aim for one workgroup per CU as well (their LDS allows no
// second): one round of workgroups, each streaming all of its chunk's tiles with the ring
// running on through the selections, instead of two rounds of half-length chunks.  Batches of
// 65 to 128 queries (one query block) take 128-row tiles, so that the chunks of a small index
// still fill every CU (32,768 rows: 256 workgroups instead of 128).
#define MF_SET(DT)                                                                              \
  MFKQI(DT, 1, 1, 16, 1, 5, 0, 1, 1, 16, 8), MFKQ(DT, 1, 1, 16, 1, 8, 0, 1, 1, 16, kWaves, 8),        \
      MFKQ(DT, 1, 1, 16, 1, 16, 0, 1, 1, 16, kWaves, 8), MF_KSI(DT, 1, 1, 16, 1, 1, 1, 16),             \
      MF_KSI(DT, 1, 1, 4, 1, 1, 1, 16), MF_KS(DT, 4, 2, 8, 1, 4, 17, 64), MF_KS(DT, 4, 2, 4, 1, 4, 17, 64), \
      MFK(DT, 8, 2, 4, 2, 5, 0, 1, 65, 128), MFK(DT, 8, 2, 4, 2, 8, 0, 1, 65, 128),                   \
      MFK(DT, 8, 2, 4, 2, 16, 0, 1, 65, 128), MFKI(DT, 8, 4, 4, 2, 5, 0, 1, 65, 1 << 30),              \
      MFK(DT, 8, 4, 4, 4, 8, 0, 1, 65, 1 << 30), MFK(DT, 8, 4, 4, 4, 16, 0, 1, 65, 1 << 30),         \
      MFK(DT, 2, 4, 8, 1, 8, 1, 4, 1, 1 << 30), MFK(DT, 2, 4, 4, 1, 8, 1, 4, 1, 1 << 30),            \
      MFKQ(DT, 1, 1, 16, 1, 5, 2, 1, 1, 16, kWaves, 8), MFK(DT, 1, 1, 16, 1, 5, 2, 8, 1, 16),          \
      MFK(DT, 1, 1, 4, 1, 5, 2, 8, 1, 16),                                                          \
      MFK(DT, 4, 2, 8, 1, 5, 2, 1, 17, 128), MFK(DT, 4, 2, 4, 1, 5, 2, 1, 17, 128),                    \
      MFKQ(DT, 8, 4, 4, 1, 5, 2, 2, 65, 1 << 30, kWaves, 3), MFK(DT, 8, 4, 4, 1, 5, 2, 2, 65, 1 << 30), \
      MFK(DT, 8, 4, 4, 1, 5, 3, 2, 1, 1 << 30), MF_DH(DT)
// The resident-query small filtered kernel (batches up to 16, and every first level) aims
// for one workgroup per CU too: 2,048 first-level rows are 16 query blocks x 16 chunks of two
// 64-row tiles, one round, instead of 512 one-tile workgroups that each load their queries.
// The 64-query filtered kernels also serve 65-128 queries (two query blocks over 128-row
// tiles keep every CU busy, where one 128-query block over 256-row tiles fills half of them),
// and aim for one workgroup per CU as well.
// Filtered kernels for levels with many hits per tile (SEL 4), one per SEL 2 shape.
#define MF_DH(DT)                                                                                          \
  MFK(DT, 1, 1, 16, 1, 5, 4, 8, 1, 16), MFK(DT, 1, 1, 4, 1, 5, 4, 8, 1, 16), MFK(DT, 4, 2, 8, 1, 5, 4, 4, 17, 128), \
      MFK(DT, 4, 2, 4, 1, 5, 4, 4, 17, 128), MFKQ(DT, 8, 4, 4, 1, 5, 4, 2, 65, 1 << 30, kWaves, 3),               \
      MFK(DT, 8, 4, 4, 1, 5, 4, 2, 65, 1 << 30)

const KernelInfo kKernels[] = {
    {dense_f32_kernel<5, 0>, kDtypeF32, 32, 64, 5, 0, 4, 1, 1 << 30, 0, kThreads, 0},
    {dense_f32_kernel<8, 0>, kDtypeF32, 32, 64, 8, 0, 4, 1, 1 << 30, 0, kThreads, 0},
    {dense_f32_kernel<16, 0>, kDtypeF32, 32, 64, 16, 0, 4, 1, 1 << 30, 0, kThreads, 0},
    {dense_f32_kernel<8, 1>, kDtypeF32, 32, 64, 128, 1, 4, 1, 1 << 30, 0, kThreads, 0},
    MF_SET(kDtypeBF16),
    MF_SET(kDtypeF16),
};
constexpr int kNumKernels = sizeof(kKernels) / sizeof(kKernels[0]);

int pick_kernel(int dtype, int d, int nq, int k, int sel) {
  const int ks = k <= 5 ? 5 : (k <= 8 ? 8 : 16);
  for (int i = 0; i < kNumKernels; ++i) {
    const KernelInfo& ki = kKernels[i];
    if (ki.dtype != dtype || ki.sel != sel) continue;
    if (sel == 0 && ki.ks != ks) continue;
    if (nq < ki.min_nq || nq > ki.max_nq) continue;
    if (ki.ring && (d / 32) % ki.ring != 0) continue;
    if (ki.qres && d / 128 > ki.qres) continue;
    return i;
  }
  return -1;
}

constexpr long long kFilterMin = 2048;        // fewest rows of a level that has a successor
constexpr long long kFilterFirstMax = 4096;   // most rows of the first level
constexpr long long kFilterLast = 16;         // row growth into the last level
constexpr long long kFilterGrow = 8;          // row growth between earlier levels
constexpr long long kFilterAllRows = 32768;   // up to this many rows a buffer holds every row

// Workgroups per query block such that the grid holds at most the kernel's target number of
// workgroups per CU (at least enough to keep every chunk of a ring kernel under 2^30 bytes of
// rows, the reach of its 32-bit offsets).  Rounding down keeps a one-per-CU grid in one round.
long long chunk_bound(const KernelInfo& ki, int d, long long n_rows, int n_qblocks, int n_cus, long long* min_chunks) {
  const long long target = (long long)n_cus * ki.chunk_target;
  long long bound = std::max(1ll, target / n_qblocks);
  long long mc = 1;
  if (ki.ring) {
    const long long n_tiles = (n_rows + ki.tile_rows - 1) / ki.tile_rows;
    const long long max_tiles = std::max(1ll, (1ll << 30) / ((long long)ki.tile_rows * d * 2));
    mc = std::max(1ll, (n_tiles + max_tiles - 1) / max_tiles);
    bound = std::max(bound, mc);
  }
  if (min_chunks) *min_chunks = mc;
  return bound;
}

// Splits n_rows into chunks (whole tiles) for one launch.
void split_rows(DensePlan& p, long long n_rows, long long chunks, long long min_chunks) {
  const long long n_tiles = (n_rows + p.tile_rows - 1) / p.tile_rows;
  chunks = std::max(min_chunks, std::max(1ll, std::min(chunks, n_tiles)));
  const long long tiles_per_chunk = n_tiles ? (n_tiles + chunks - 1) / chunks : 1;
  p.rows_per_chunk = tiles_per_chunk * p.tile_rows;
  p.n_chunks = (int)std::max(1ll, n_tiles ? (n_tiles + tiles_per_chunk - 1) / tiles_per_chunk : 1);
  p.grid = (long long)p.n_chunks * p.n_qblocks;
}

size_t align_up256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

DensePlan plan_dense_lists(int dtype, int d, long long n_rows, int nq, int k, int n_cus) {
  DensePlan p;
  p.n_cus = n_cus;
  p.kernel = pick_kernel(dtype, d, nq, k, k <= 16 ? 0 : 1);
  if (p.kernel < 0) return p;
  const KernelInfo& ki = kKernels[p.kernel];
  p.bn = ki.bn;
  p.tile_rows = ki.tile_rows;
  p.n_qblocks = (nq + p.bn - 1) / p.bn;
  long long min_chunks = 1;
  const long long bound = chunk_bound(ki, d, n_rows, p.n_qblocks, n_cus, &min_chunks);
  const long long n_tiles = (n_rows + p.tile_rows - 1) / p.tile_rows;
  long long chunks = bound;
  // the queue-based large-k selector wants several tiles per chunk so its queues amortise
  if (ki.sel == 1) chunks = std::min(chunks, std::max(1ll, n_tiles / 4));
  split_rows(p, n_rows, chunks, min_chunks);
  p.cap = bound * k;  // partial slots per query for any row count (n_chunks <= bound)
  return p;
}

DensePlan plan_dense(int dtype, int d, long long n_rows, int nq, int k, int n_cus) {
  if (dtype == kDtypeF32 || k <= 16) return plan_dense_lists(dtype, d, n_rows, nq, k, n_cus);
  DensePlan p;
  p.n_cus = n_cus;
  p.kernel = pick_kernel(dtype, d, nq, k, 2);
  if (p.kernel < 0) return plan_dense_lists(dtype, d, n_rows, nq, k, n_cus);
  const KernelInfo& ki = kKernels[p.kernel];
  p.filtered = true;
  p.bn = ki.bn;
  p.tile_rows = ki.tile_rows;
  p.n_qblocks = (nq + p.bn - 1) / p.bn;
  // Levels: row prefixes, each filtered by the previous level's k-th score; the first takes
  // every score as a candidate, the last is all rows.  Built from the end: the level before
  // the last holds n_rows / kFilterLast rows (the last level, the one that streams the whole
  // index, then admits about k * kFilterLast rows per query), earlier ones shrink
  // kFilterGrow-fold (to no fewer than kFilterMin rows) until the first has at most
  // kFilterFirstMax.  A level expects at most about k * max(kFilterGrow, kFilterLast)
  // candidates per query; fcap allows four times that, and the whole first level.  Up to
  // kFilterAllRows rows a buffer holds every row (at most 256 KB per query), so no level can
  // overflow and the repair launches are left out.
  long long back[8];
  int nb = 0;
  back[nb++] = n_rows;
  {
    long long r = std::max(kFilterMin, (n_rows + kFilterLast - 1) / kFilterLast);
    // One level over all rows where it costs less: a short index, or up to 64 queries over at
    // most kFilterAllRows rows (the threshold level and its selection cost two launches, more
    // than ranking every row's key: batch 1 top-100 over 32,768 rows 36.7 -> 34.2 us per call,
    // batch 64 45.3 -> 44.2; above 64 queries the levels stay ahead).
    if (4 * r <= n_rows && !(nq <= 64 && n_rows <= kFilterAllRows)) {
      back[nb++] = r;
      while (nb < 8 && r > kFilterFirstMax) {
        r = std::max(kFilterMin, (r + kFilterGrow - 1) / kFilterGrow);
        back[nb++] = r;
      }
    }
  }
  p.n_levels = nb;
  for (int l = 0; l < nb; ++l) p.level_rows[l] = back[nb - 1 - l];
  p.fcap = n_rows <= kFilterAllRows
               ? std::max(1ll, n_rows)
               : std::max(1ll, std::min(n_rows, std::max(p.level_rows[0],
                                                         4 * std::max(kFilterGrow, kFilterLast) * (long long)k)));
  p.repair = p.fcap < n_rows;
  p.chunk_bound = chunk_bound(ki, d, n_rows, p.n_qblocks, n_cus, nullptr);
  p.kernel0 = p.kernel;
  p.n_qblocks0 = p.n_qblocks;
  p.chunk_bound0 = p.chunk_bound;
  {
    DensePlan l0 = p;
    split_rows(l0, p.level_rows[0], p.chunk_bound, 1);
    const int small = pick_kernel(dtype, d, 1, k, 2);
    if (l0.grid < n_cus && small >= 0) {  // the main kernel would leave most CUs idle
      const KernelInfo& ks = kKernels[small];
      p.kernel0 = small;
      p.n_qblocks0 = (nq + ks.bn - 1) / ks.bn;
      p.chunk_bound0 = chunk_bound(ks, d, p.level_rows[0], p.n_qblocks0, n_cus, nullptr);
    }
  }
  split_rows(p, n_rows, p.chunk_bound, 1);
  // the per-chunk-list plan is the exact fallback; the workspace covers it as well
  p.cap = plan_dense_lists(dtype, d, n_rows, nq, k, n_cus).cap;
  return p;
}

// Filtered-mode workspace: candidate buffers [nq][fcap] | counts [nq] | (shared with the
// per-chunk lists of the fallback plan) | four overflow flags past both.
namespace {
size_t filtered_body_bytes(const DensePlan& p, int nq) {
  const size_t lists = (size_t)nq * (size_t)p.cap * sizeof(unsigned long long);
  const size_t filt = align_up256((size_t)nq * (size_t)p.fcap * 8) + align_up256((size_t)nq * 4);
  return align_up256(std::max(lists, filt));
}
// [0] the last level overflowed, [1] an earlier level did (harmless), [2] the repair did.
int* dense_flags(const DensePlan& p, void* ws, int nq) {
  return reinterpret_cast<int*>(static_cast<unsigned char*>(ws) + filtered_body_bytes(p, nq));
}
}  // namespace

size_t dense_workspace_bytes(const DensePlan& p, int nq) {
  if (!p.filtered) return (size_t)nq * (size_t)p.cap * sizeof(unsigned long long);
  return filtered_body_bytes(p, nq) + 256;
}

// The plan's workspace grows with the row count except where buffers stop holding every row
// (fcap drops from kFilterAllRows to max(kFilterFirstMax, 256 k)), so the bound over all row
// counts up to `capacity` is the larger of the two plans on either side.
size_t dense_workspace_bound(int dtype, int d, long long capacity, int nq, int k, int n_cus) {
  size_t b = dense_workspace_bytes(plan_dense(dtype, d, capacity, nq, k, n_cus), nq);
  if (capacity > kFilterAllRows)
    b = std::max(b, dense_workspace_bytes(plan_dense(dtype, d, kFilterAllRows, nq, k, n_cus), nq));
  return b;
}

namespace {

hipError_t launch_kernel(const KernelInfo& ki, long long grid, DenseArgs& arg, hipStream_t s, hipEvent_t ev0,
                         hipEvent_t ev1) {
  void* params[] = {&arg};
  // With timing events the launch carries them in its dispatch packet: they are stamped when
  // the kernel itself starts and ends.
  return ev0 ? hipExtLaunchKernel(reinterpret_cast<const void*>(ki.fn), dim3((unsigned)grid), dim3(ki.threads), params,
                                  0, s, ev0, ev1, 0)
             : hipLaunchKernel(reinterpret_cast<const void*>(ki.fn), dim3((unsigned)grid), dim3(ki.threads), params, 0,
                               s);
}

// The many-hits variant (SEL 4) of filtered kernel i: the same shape, or i itself.
int dense_hits_twin(int i) {
  const KernelInfo& a = kKernels[i];
  for (int j = 0; j < kNumKernels; ++j) {
    const KernelInfo& b = kKernels[j];
    if (b.sel == 4 && b.dtype == a.dtype && b.bn == a.bn && b.tile_rows == a.tile_rows && b.ring == a.ring &&
        b.threads == a.threads && b.qres == a.qres && b.min_nq == a.min_nq && b.max_nq == a.max_nq)
      return j;
  }
  return i;
}

// Exact top-k of each query's candidate buffer (threshold_only: just a valid k-th score).
void launch_select(int n_cus, const unsigned long long* cbuf, int* ccnt, long long cap, int nq, int k, float* out_scores,
                   long long* out_ids, int* ovf, const int* gate, bool threshold_only, hipStream_t s) {
  if (nq <= 2 * n_cus)
    hipLaunchKernelGGL(select_topk_kernel<1024>, dim3((unsigned)nq), dim3(1024), 0, s, cbuf, ccnt, cap, k, out_scores,
                       out_ids, ovf, gate, threshold_only ? 1 : 0);
  else
    hipLaunchKernelGGL(select_topk_kernel<256>, dim3((unsigned)nq), dim3(256), 0, s, cbuf, ccnt, cap, k, out_scores,
                       out_ids, ovf, gate, threshold_only ? 1 : 0);
}

// One filter pass over rows [0, rows): candidates >= th (every row when th is null) into the
// buffers, then the exact top-k of each buffer (threshold_only: just a valid k-th score for
// the next level).  The first pass (th null) sets the counts; each selection zeroes its
// query's count for the next pass.  prev_rows: the rows of the prefix th comes from (about
// k / prev_rows of the rows are hits).  With a gate, nothing runs unless *gate != 0.
hipError_t filter_pass(const DensePlan& p, const DenseArgs& a, long long rows, const float* th, long long prev_rows,
                       int* ovf, const int* gate, bool threshold_only, bool first, hipStream_t s, hipEvent_t ev0,
                       hipEvent_t ev1) {
  // about k / prev_rows of the rows are hits: from 1 in 64 on, the many-hits variant
  const int kidx = first ? p.kernel0 : p.kernel;
  const KernelInfo& ki = kKernels[th != nullptr && 64ll * a.k >= prev_rows ? dense_hits_twin(kidx) : kidx];
  unsigned long long* cbuf = a.partial;  // the workspace
  int* ccnt = reinterpret_cast<int*>(reinterpret_cast<unsigned char*>(cbuf) +
                                     align_up256((size_t)a.nq * (size_t)p.fcap * 8));
  DensePlan lp = p;
  lp.tile_rows = ki.tile_rows;
  lp.n_qblocks = first ? p.n_qblocks0 : p.n_qblocks;
  split_rows(lp, rows, first ? p.chunk_bound0 : p.chunk_bound, 1);
  DenseArgs arg = a;
  arg.n_qblocks = lp.n_qblocks;
  arg.n_rows = rows;
  arg.n_chunks = lp.n_chunks;
  arg.rows_per_chunk = lp.rows_per_chunk;
  arg.th = th;
  arg.th_stride = a.k;
  arg.cbuf = cbuf;
  arg.ccnt = ccnt;
  arg.cap = p.fcap;
  arg.gate = gate;
  hipError_t e = launch_kernel(ki, lp.grid, arg, s, ev0, ev1);
  if (e != hipSuccess) return e;
  launch_select(p.n_cus, cbuf, ccnt, p.fcap, a.nq, a.k, a.out_scores, a.out_ids, ovf, gate, threshold_only, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_dense(const DensePlan& p, int dtype, const DenseArgs& a, hipStream_t s, hipEvent_t ev0,
                        hipEvent_t ev1) {
  const KernelInfo& ki = kKernels[p.kernel];
  if (p.filtered) {
    // The overflow flags matter only where a buffer can overflow; otherwise no flag is
    // passed, and there is nothing to clear.
    int* fl = p.repair ? dense_flags(p, a.partial, a.nq) : nullptr;
    if (p.repair) hipLaunchKernelGGL(clear_ints_kernel, dim3(1), dim3(64), 0, s, fl, 4ll, nullptr);
    for (int l = 0; l < p.n_levels; ++l) {
      const bool last = l == p.n_levels - 1;
      // level l's threshold: a lower bound of the k-th score over level l - 1's rows
      hipError_t e = filter_pass(p, a, p.level_rows[l], l == 0 ? nullptr : a.out_scores + (a.k - 1),
                                 l == 0 ? 0 : p.level_rows[l - 1], fl ? fl + (last ? 0 : 1) : nullptr,
                                 nullptr, !last, l == 0, s, last ? ev0 : nullptr, last ? ev1 : nullptr);
      if (e != hipSuccess) return e;
    }
    if (!p.repair) return hipGetLastError();  // every buffer holds all rows: nothing can overflow
    // Exactness repair, decided on the device: only a buffer overflow in the last level can
    // lose a row.  Then the last level runs again with the current k-th scores as thresholds
    // (the lists are the top-k of a subset of the rows at or above the old thresholds, so
    // their k-th scores are valid thresholds and no lower), and if that overflows too, the
    // per-chunk-list plan runs.  Each repair launch returns at once when its flag is clear.
    hipError_t e =
        filter_pass(p, a, a.n_rows, a.out_scores + (a.k - 1), a.n_rows, fl + 2, fl, false, false, s, nullptr, nullptr);
    if (e != hipSuccess) return e;
    const DensePlan lp = plan_dense_lists(dtype, a.d, a.n_rows, a.nq, a.k, p.n_cus);
    DenseArgs la = a;
    la.n_qblocks = lp.n_qblocks;
    la.n_chunks = lp.n_chunks;
    la.rows_per_chunk = lp.rows_per_chunk;
    la.gate = fl + 2;
    const KernelInfo& lk = kKernels[lp.kernel];
    e = launch_kernel(lk, lp.grid, la, s, nullptr, nullptr);
    if (e != hipSuccess) return e;
    if (lp.n_chunks > 1)
      hipLaunchKernelGGL(merge_large_kernel, dim3((unsigned)((a.nq + kWaves - 1) / kWaves)), dim3(kThreads), 0, s,
                         a.partial, lp.n_chunks, a.nq, a.k, a.out_scores, a.out_ids, fl + 2);
    return hipGetLastError();
  }
  DenseArgs arg = a;
  hipError_t e = launch_kernel(ki, p.grid, arg, s, ev0, ev1);
  if (e != hipSuccess || p.n_chunks == 1) return e;
  if (ki.sel == 0) {
    // one batch of 16 composites per lane where the lists fit it, else 32 (the 256 five-entry
    // lists of a small batch then still fit one), else a workgroup per query
    const long long nc = (long long)p.n_chunks * a.k;
    const dim3 mg((unsigned)((a.nq + kWaves - 1) / kWaves));
    if (nc <= 64 * 16)
      hipLaunchKernelGGL(merge_lists_kernel<16>, mg, dim3(kThreads), 0, s, a.partial, p.n_chunks, a.nq, a.k,
                         a.out_scores, a.out_ids);
    else if (nc <= 64 * 32)
      hipLaunchKernelGGL(merge_lists_kernel<32>, mg, dim3(kThreads), 0, s, a.partial, p.n_chunks, a.nq, a.k,
                         a.out_scores, a.out_ids);
    else  // the list kernels have k <= 16 = kWgMergeK
      hipLaunchKernelGGL(merge_lists_wg_kernel, dim3((unsigned)a.nq), dim3(kThreads), 0, s, a.partial, p.n_chunks,
                         a.nq, a.k, a.out_scores, a.out_ids);
  } else {
    hipLaunchKernelGGL(merge_large_kernel, dim3((unsigned)((a.nq + kWaves - 1) / kWaves)), dim3(kThreads), 0, s,
                       a.partial, p.n_chunks, a.nq, a.k, a.out_scores, a.out_ids, nullptr);
  }
  return hipGetLastError();
}


DensePlan plan_dense_dump(int dtype, int d, long long n_rows, int nq, int n_cus) {
  DensePlan p;
  p.n_cus = n_cus;
  p.kernel = pick_kernel(dtype, d, nq, 5, 3);
  if (p.kernel < 0) return p;
  const KernelInfo& ki = kKernels[p.kernel];
  p.bn = ki.bn;
  p.tile_rows = ki.tile_rows;
  p.n_qblocks = (nq + p.bn - 1) / p.bn;
  long long mc = 1;
  const long long bound = chunk_bound(ki, d, n_rows, p.n_qblocks, n_cus, &mc);
  split_rows(p, n_rows, bound, mc);
  return p;
}

hipError_t launch_dense_dump(const DensePlan& p, const DenseArgs& a, hipStream_t s) {
  DenseArgs arg = a;
  arg.n_qblocks = p.n_qblocks;
  arg.n_chunks = p.n_chunks;
  arg.rows_per_chunk = p.rows_per_chunk;
  return launch_kernel(kKernels[p.kernel], p.grid, arg, s, nullptr, nullptr);
}

hipError_t launch_weighted_fuse(int n_cus, const float* D, const float* B, long long ld, long long n, long long n_lex, int nq,
                                const float* mm_d, int pd, const float* mm_l, int pl, double wd, double wl, int k,
                                unsigned long long* cbuf, int* ccnt, float* out_scores, long long* out_ids,
                                hipStream_t s) {
  hipLaunchKernelGGL(weighted_fuse_kernel, dim3((unsigned)nq), dim3(kFuseThreads), 0, s, D, B, ld, n, n_lex, mm_d, pd,
                     mm_l, pl, wd, wl, k, cbuf, ccnt);
  launch_select(n_cus, cbuf, ccnt, n, nq, k, out_scores, out_ids, nullptr, nullptr, false, s);
  return hipGetLastError();
}

}  // namespace oprag
#endif  // OPRAG_DENSE_ILP
