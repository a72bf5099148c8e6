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
// Data movement for bf16 / fp16: each stage of KC = 64 dimensions is copied straight from
// global memory into an LDS ring slot with global_load_lds_dwordx4 (no VGPR round trip),
// already in MFMA fragment order (one 1 KiB fragment = 16 rows x 32 dims, lane i's 16 bytes
// at offset 16 i), so every fragment read is a linear, conflict-free ds_read_b128.  The
// waves form a WM x WN grid over (rows x queries); each loads the fragments of a 32-dim step
// for its subtile before issuing that step's MFMAs, and the next step's fragments while the
// MFMAs run.
//
// Selection (k <= 16): per tile, the score subtile goes to LDS query-major.  Pass 1 keeps the
// top-KS *values* of each thread's row slice with a branch-free v_med3 insertion network
// (one instruction per slot), and the values are combined per query with the running list
// to give the k-th best value tau.  Pass 2 appends only rows scoring above tau, plus the
// smallest-id rows equal to tau that may still be needed, to a small per-query candidate
// list, which the query's owner thread inserts into its running (score desc, id asc) list.
// Exact, and the 64-bit composite compares run on at most 2k - 1 candidates per query and
// pass.  Selection (k <= 128): one wave per query keeps a 128-entry sorted queue and merges
// batches of 64 candidates above its k-th entry with a bitonic network.
#include <algorithm>

#include "oprag_internal.h"
#include "select.h"

namespace oprag {
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

#define OPRAG_LDS(p) ((__attribute__((address_space(3))) void*)(p))

// 16 bytes per lane, global -> LDS; lane i's bytes land at lds_base + 16 * i.
__device__ __forceinline__ void dma16(const void* g, void* lds_base) {
  __builtin_amdgcn_global_load_lds(g, OPRAG_LDS(lds_base), 16, 0, 0);
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
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
template <int BN, int KS>
struct SelSmall {
  static constexpr int TPQ = kThreads / BN;  // threads per query: t = q + BN * sub
  static constexpr int CAP = 2 * KS > 16 ? 2 * KS : 16;  // candidate slots per query and pass
  static constexpr int NL = KS <= 8 ? 4 : 2;             // independent value lists per thread
  static constexpr int kVals = TPQ > 1 ? TPQ * BN * KS * 4 : 0;
  static constexpr int kBytes = BN * CAP * 8 + kVals + TPQ * BN * 4 + BN * 12 + 16;
  RegTopK<KS> run;  // running list of the query (owner thread, sub == 0)

  __device__ __forceinline__ void init() { run.clear(); }

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

template <int BN, int KS, int SEL>
struct SelOf {
  typedef SelSmall<BN, KS> type;
};
template <int BN, int KS>
struct SelOf<BN, KS, 1> {
  typedef SelLarge<BN> type;
};

// ------------------------------------------------------------------------------------
// bf16 / fp16 MFMA kernel.  Four waves split a tile of TR = 4*MW*16 rows (each wave owns
// MW distinct 16-row subtiles) and share a block of BN = NW*16 queries.  Stages are 32
// dimensions.  Row fragments go global -> VGPRs directly in MFMA A-operand layout (each
// wave reads only its own rows, no LDS); query pieces go global -> VGPRs -> an LDS slot
// (double-buffered) from which every wave reads its B operands.  Both sit in a register
// ring of RS stages issued PX = RS - 1 stages ahead; the stage loop runs across the tiles
// of the chunk, so the next tile's loads are in flight while a tile's selection runs.
// The epilogue takes G passes of MW/G subtiles per wave through the LDS score tile.
// ------------------------------------------------------------------------------------
template <int DT, int NW, int MW, int RS, int G, int KS, int SEL>
__global__ __launch_bounds__(kThreads) void dense_mfma_kernel(DenseArgs a) {
  using M = Mfma<DT>;
  using V = typename M::V;
  using T = typename M::T;
  constexpr int BN = NW * 16;
  constexpr int TR = kWaves * MW * 16;
  constexpr int KC = 32;
  constexpr int PX = RS - 1;
  constexpr int QSLOT = BN * KC * 2;            // bytes; a query row is 4 pieces of 16 bytes
  constexpr int QPC = BN * KC * 2 / 16;         // 16-byte query pieces per stage
  constexpr int QPT = (QPC + kThreads - 1) / kThreads;
  constexpr int MWP = MW / G;                   // subtile rows per wave per pass
  constexpr int RP = kWaves * MWP * 16;         // rows per pass
  constexpr int SR = RP + 4;                    // S row stride (floats)
  using Sel = typename SelOf<BN, KS, SEL>::type;
  constexpr int QBYTES = 2 * QSLOT;
  constexpr int SBYTES = BN * SR * 4;
  constexpr int SMEM = QBYTES + SBYTES + Sel::kBytes;
  static_assert(MW % G == 0 && ((MWP * 16) & (MWP * 16 - 1)) == 0, "pass shape");
  static_assert(SEL == 1 || RP % (4 * (kThreads / BN)) == 0, "slice shape");
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
  const int nk = d / KC;                                            // stages per tile
  const int n_tiles = (int)((row_end - row_begin + TR - 1) / TR);   // 0 for an empty chunk
  const int n_st = n_tiles * nk;
  const T* X = static_cast<const T*>(a.X);
  const T* Q = static_cast<const T*>(a.Q);
  const int kl = (lane >> 4) * 8;  // this lane's 8 dimensions inside a 32-dim stage

  // query pieces of this thread: piece p -> query row r = p / 4, 16-byte column cc = p % 4,
  // stored at column (cc + r / 2) % 4 of the row: any 8 consecutive lanes then touch 128
  // distinct bytes modulo 128, both for the row-wise writes and for the fragment reads
  // (8 rows, one column).  When a stage has fewer
  // pieces than threads, several threads copy the same piece (identical bytes, same place),
  // so every load and store is unconditional.
  const T* qsrc[QPT];
  int qdst[QPT];
#pragma unroll
  for (int j = 0; j < QPT; ++j) {
    const int p = (tid + kThreads * j) % QPC;
    const int r = p / (KC / 8), cc = p % (KC / 8);
    qsrc[j] = Q + (long long)min(q0 + r, a.nq - 1) * d + cc * 8;
    qdst[j] = r * 64 + ((cc + (r >> 1)) & 3) * 16;
  }
  const int xrow0 = w * MW * 16 + (lane & 15);  // row of subtile 0 inside a tile
  int fbo[NW];  // byte offset of this lane's B-fragment piece in a query slot
#pragma unroll
  for (int ni = 0; ni < NW; ++ni) {
    const int n = ni * 16 + (lane & 15);
    fbo[ni] = n * 64 + (((lane >> 4) + (n >> 1)) & 3) * 16;
  }

  // Register ring of RS = 4 stages; every index below is a literal so the ring stays in VGPRs.
  static_assert(RS == 4, "the stage loop below is written out for a ring of 4");
  V xr[RS][MW];
  u32x4 qr[RS][QPT];
#define OPRAG_ISSUE(GS, SLOT)                                                            \
  {                                                                                      \
    const int t_ = (GS) / nk, c_ = (GS) - t_ * nk;                                       \
    const long long tile0_ = row_begin + (long long)t_ * TR;                             \
    _Pragma("unroll") for (int mi = 0; mi < MW; ++mi) {                                  \
      const long long row_ = min(tile0_ + xrow0 + mi * 16, a.n_rows - 1);               \
      xr[SLOT][mi] = *reinterpret_cast<const V*>(X + row_ * d + c_ * KC + kl);           \
    }                                                                                    \
    _Pragma("unroll") for (int j = 0; j < QPT; ++j) qr[SLOT][j] =                        \
        *reinterpret_cast<const u32x4*>(qsrc[j] + c_ * KC);                              \
  }
#define OPRAG_STEP(U)                                                                    \
  if (gs0 + (U) < n_st) {                                                                \
    const int gs = gs0 + (U);                                                            \
    if (gs + PX < n_st) OPRAG_ISSUE(gs + PX, ((U) + PX) % RS);                           \
    unsigned char* qs = qslots + (gs & 1) * QSLOT;                                       \
    _Pragma("unroll") for (int j = 0; j < QPT; ++j)                                      \
        *reinterpret_cast<u32x4*>(qs + qdst[j]) = qr[U][j];                              \
    lds_barrier();                                                                       \
    V fb[NW];                                                                            \
    _Pragma("unroll") for (int ni = 0; ni < NW; ++ni) fb[ni] =                           \
        *reinterpret_cast<const V*>(qs + fbo[ni]);                                       \
    _Pragma("unroll") for (int ni = 0; ni < NW; ++ni)                                    \
        _Pragma("unroll") for (int mi = 0; mi < MW; ++mi)                                \
            acc[mi][ni] = M::run(xr[U][mi], fb[ni], acc[mi][ni]);                        \
  }

  Sel sel;
  sel.init();
  f32x4 acc[MW][NW];
#pragma unroll
  for (int mi = 0; mi < MW; ++mi)
#pragma unroll
    for (int ni = 0; ni < NW; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (0 < n_st) OPRAG_ISSUE(0, 0);
  if (1 < n_st) OPRAG_ISSUE(1, 1);
  if (2 < n_st) OPRAG_ISSUE(2, 2);

  for (int gs0 = 0; gs0 < n_st; gs0 += RS) {
    // d % 128 == 0 makes nk a multiple of RS, so every group of RS stages lies in one tile
    OPRAG_STEP(0)
    OPRAG_STEP(1)
    OPRAG_STEP(2)
    OPRAG_STEP(3)
    if ((gs0 + RS) % nk == 0) {
      // ---- epilogue of the tile: G passes through the query-major LDS score tile
      const long long tile0 = row_begin + (long long)(gs0 / nk) * TR;
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
        for (int bb = 0; bb < kWaves; ++bb) {
          const long long start = tile0 + (long long)bb * MW * 16 + g * MWP * 16;
          nv += (int)max(0ll, min((long long)(MWP * 16), row_end - start));
        }
        pr.nvalid = nv;
        lds_barrier();
        sel.pass(S, SR, RP, pr, q_lim, a.k, scratch);
      }
#pragma unroll
      for (int mi = 0; mi < MW; ++mi)
#pragma unroll
        for (int ni = 0; ni < NW; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
#undef OPRAG_STEP
#undef OPRAG_ISSUE
  sel.write(a, q0, chunk);
}

// ------------------------------------------------------------------------------------
// fp32 VALU kernel: tile of 64 rows x 32 queries, 32 dimensions per stage.
// ------------------------------------------------------------------------------------
template <int KS, int SEL>
__global__ __launch_bounds__(kThreads) void dense_f32_kernel(DenseArgs a) {
  constexpr int BN = 32, TR = 64, KC = 32, SR = TR + 4;
  using Sel = typename SelOf<BN, KS, SEL>::type;
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

  for (long long tile0 = row_begin; tile0 < row_end; tile0 += TR) {
    float acc[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) acc[r] = 0.f;
    for (int kc = 0; kc < d; kc += KC) {
      __syncthreads();
      for (int i = tid; i < TR * KC; i += kThreads) {
        const int r = i / KC, c = i % KC;
        const long long row = min(tile0 + r, a.n_rows - 1);
        Xs[r * (KC + 1) + c] = (kc + c < d) ? X[row * d + kc + c] : 0.f;
      }
      for (int i = tid; i < BN * KC; i += kThreads) {
        const int r = i / KC, c = i % KC;
        const int qr = min(q0 + r, a.nq - 1);
        Qs[r * (KC + 1) + c] = (kc + c < d) ? Q[(long long)qr * d + kc + c] : 0.f;
      }
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
// Merge of the per-chunk lists: partial[q][chunk][k] composites (0 = empty slot).
// ------------------------------------------------------------------------------------
// k <= KS <= 16: one workgroup per query.  Thread t owns a contiguous block of the query's
// candidates (chunk lists in row order, each sorted), so thread order is id order among
// equal scores.  Pass 1: top-KS values per thread (med3), combined across the wave with
// shuffles and across waves through LDS into the exact k-th value tau.  Pass 2: candidates
// above tau and the first (smallest-id) ones equal to tau go to LDS; thread 0 sorts them.
template <int KS>
__global__ __launch_bounds__(kThreads) void merge_small_kernel(const unsigned long long* __restrict__ partial,
                                                               int n_chunks, int nq, int k, float* out_scores,
                                                               long long* out_ids) {
  constexpr int CAP = 2 * KS;
  __shared__ u64 cand[CAP];
  __shared__ float wl[kWaves][KS];
  __shared__ int wsum[kWaves];
  __shared__ float s_tau;
  __shared__ int s_need, s_cnt;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int q = blockIdx.x;
  const long long n = (long long)n_chunks * k;
  const int per = (int)((n + kThreads - 1) / kThreads);
  const long long b0 = (long long)t * per;
  const long long b1 = b0 + per < n ? b0 + per : n;
  const unsigned long long* src = partial + (long long)q * n;

  ValTop<KS> L;
  L.clear();
  for (long long j = b0; j < b1; j += 4) {
    u64 c[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) c[u] = j + u < b1 ? src[j + u] : 0ull;
#pragma unroll
    for (int u = 0; u < 4; ++u) L.insert(c[u] ? comp_score(c[u]) : kNegInf);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    float o[KS];
#pragma unroll
    for (int i = 0; i < KS; ++i) o[i] = __shfl_xor(L.v[i], off, 64);
#pragma unroll
    for (int i = 0; i < KS; ++i) L.insert(o[i]);
  }
  if (lane == 0)
#pragma unroll
    for (int i = 0; i < KS; ++i) wl[w][i] = L.v[i];
  if (t == 0) s_cnt = 0;
  __syncthreads();
  if (t == 0) {
    for (int ww = 1; ww < kWaves; ++ww)
#pragma unroll
      for (int i = 0; i < KS; ++i) L.insert(wl[ww][i]);
    const float tau = L.at(k);
    int ngt = 0;
#pragma unroll
    for (int i = 0; i < KS; ++i) ngt += (i < k && L.v[i] > tau) ? 1 : 0;
    s_tau = tau;
    s_need = tau == kNegInf ? 0 : k - ngt;
  }
  __syncthreads();
  const float tau = s_tau;
  const int need = s_need;
  int neq = 0;
  for (long long j = b0; j < b1; ++j) {
    const u64 c = src[j];
    if (!c) continue;
    const float v = comp_score(c);
    if (v > tau) cand[atomicAdd(&s_cnt, 1)] = c;
    neq += v == tau ? 1 : 0;
  }
  // exclusive prefix of the tie counts in thread order
  int x = neq;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  int pre = x - neq;
  for (int ww = 0; ww < w; ++ww) pre += wsum[ww];
  if (neq > 0 && pre < need)
    for (long long j = b0; j < b1 && pre < need; ++j) {
      const u64 c = src[j];
      if (c && comp_score(c) == tau) {
        cand[atomicAdd(&s_cnt, 1)] = c;
        ++pre;
      }
    }
  __syncthreads();
  if (t == 0) {
    RegTopK<KS> list;
    list.clear();
    for (int j = 0; j < s_cnt; ++j) list.insert(cand[j]);
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      if (i < k) {
        const u64 c = list.v[i];
        out_ids[(long long)q * k + i] = c ? (long long)comp_row(c) : -1ll;
        out_scores[(long long)q * k + i] = c ? comp_score(c) : kNegInf;
      }
    }
  }
}

// k <= 128: one wave per query keeps a 128-entry queue and merges 64 candidates at a time.
__global__ __launch_bounds__(kThreads) void merge_large_kernel(const unsigned long long* __restrict__ partial,
                                                               int n_chunks, int nq, int k, float* out_scores,
                                                               long long* out_ids) {
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
  int dtype, bn, tile_rows, ks, sel, wgs_per_cu, min_nq, max_nq;
};

#define MFK(DT, NW, MW, RS, G, KS, SEL, OCC, LO, HI) \
  {dense_mfma_kernel<DT, NW, MW, RS, G, KS, SEL>, DT, NW * 16, kWaves * MW * 16, KS, SEL, OCC, LO, HI}
#define MF_SET(DT)                                                                              \
  MFK(DT, 1, 1, 4, 1, 5, 0, 4, 1, 16), MFK(DT, 1, 1, 4, 1, 8, 0, 4, 1, 16),                    \
      MFK(DT, 1, 1, 4, 1, 16, 0, 4, 1, 16), MFK(DT, 4, 2, 4, 1, 5, 0, 2, 17, 64),              \
      MFK(DT, 4, 2, 4, 1, 8, 0, 2, 17, 64), MFK(DT, 4, 2, 4, 1, 16, 0, 2, 17, 64),             \
      MFK(DT, 8, 4, 4, 4, 5, 0, 1, 65, 1 << 30), MFK(DT, 8, 4, 4, 4, 8, 0, 1, 65, 1 << 30),    \
      MFK(DT, 8, 4, 4, 4, 16, 0, 1, 65, 1 << 30), MFK(DT, 2, 4, 4, 1, 8, 1, 2, 1, 1 << 30)

const KernelInfo kKernels[] = {
    {dense_f32_kernel<5, 0>, kDtypeF32, 32, 64, 5, 0, 2, 1, 1 << 30},
    {dense_f32_kernel<8, 0>, kDtypeF32, 32, 64, 8, 0, 2, 1, 1 << 30},
    {dense_f32_kernel<16, 0>, kDtypeF32, 32, 64, 16, 0, 2, 1, 1 << 30},
    {dense_f32_kernel<8, 1>, kDtypeF32, 32, 64, 128, 1, 2, 1, 1 << 30},
    MF_SET(kDtypeBF16),
    MF_SET(kDtypeF16),
};
constexpr int kNumKernels = sizeof(kKernels) / sizeof(kKernels[0]);

int pick_kernel(int dtype, int nq, int k) {
  const int sel = k <= 16 ? 0 : 1;
  const int ks = k <= 5 ? 5 : (k <= 8 ? 8 : 16);
  for (int i = 0; i < kNumKernels; ++i) {
    const KernelInfo& ki = kKernels[i];
    if (ki.dtype != dtype || ki.sel != sel) continue;
    if (sel == 0 && ki.ks != ks) continue;
    if (nq < ki.min_nq || nq > ki.max_nq) continue;
    return i;
  }
  return -1;
}

}  // namespace

constexpr int kNumCUs = 256;

DensePlan plan_dense(int dtype, int d, long long n_rows, int nq, int k) {
  (void)d;
  DensePlan p;
  p.kernel = pick_kernel(dtype, nq, k);
  if (p.kernel < 0) return p;
  const KernelInfo& ki = kKernels[p.kernel];
  p.bn = ki.bn;
  p.tile_rows = ki.tile_rows;
  p.n_qblocks = (nq + p.bn - 1) / p.bn;
  const long long n_tiles = (n_rows + p.tile_rows - 1) / p.tile_rows;
  // Enough workgroups to fill the chip twice over, never more chunks than tiles; the large-k
  // selector wants several tiles per chunk so its queues amortise.
  const long long target = (long long)kNumCUs * ki.wgs_per_cu * 2;
  const long long bound = std::max(1ll, (target + p.n_qblocks - 1) / p.n_qblocks);
  long long chunks = bound;
  if (ki.sel == 1) chunks = std::min(chunks, std::max(1ll, n_tiles / 4));
  chunks = std::max(1ll, std::min(chunks, n_tiles));
  const long long tiles_per_chunk = n_tiles ? (n_tiles + chunks - 1) / chunks : 1;
  p.rows_per_chunk = tiles_per_chunk * p.tile_rows;
  p.n_chunks = (int)std::max(1ll, n_tiles ? (n_tiles + tiles_per_chunk - 1) / tiles_per_chunk : 1);
  p.cap = bound * k;  // partial slots per query for any row count (n_chunks <= bound)
  p.grid = (long long)p.n_chunks * p.n_qblocks;
  return p;
}

size_t dense_workspace_bytes(const DensePlan& p, int nq) {
  return (size_t)nq * (size_t)p.cap * sizeof(unsigned long long);
}

hipError_t launch_dense(const DensePlan& p, int dtype, const DenseArgs& a, hipStream_t s) {
  (void)dtype;
  const KernelInfo& ki = kKernels[p.kernel];
  DenseArgs arg = a;
  void* params[] = {&arg};
  hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(ki.fn), dim3((unsigned)p.grid), dim3(kThreads), params,
                                 0, s);
  if (e != hipSuccess || p.n_chunks == 1) return e;
  if (ki.sel == 0) {
    const unsigned blocks = (unsigned)a.nq;
    if (ki.ks == 5)
      hipLaunchKernelGGL(merge_small_kernel<5>, dim3(blocks), dim3(kThreads), 0, s, a.partial, p.n_chunks, a.nq, a.k,
                         a.out_scores, a.out_ids);
    else if (ki.ks == 8)
      hipLaunchKernelGGL(merge_small_kernel<8>, dim3(blocks), dim3(kThreads), 0, s, a.partial, p.n_chunks, a.nq, a.k,
                         a.out_scores, a.out_ids);
    else
      hipLaunchKernelGGL(merge_small_kernel<16>, dim3(blocks), dim3(kThreads), 0, s, a.partial, p.n_chunks, a.nq,
                         a.k, a.out_scores, a.out_ids);
  } else {
    hipLaunchKernelGGL(merge_large_kernel, dim3((unsigned)((a.nq + kWaves - 1) / kWaves)), dim3(kThreads), 0, s,
                       a.partial, p.n_chunks, a.nq, a.k, a.out_scores, a.out_ids);
  }
  return hipGetLastError();
}

}  // namespace oprag
