// Dense exact top-k: R_k = Op_retrieve(q, I) (Section 3.2, "Retrieval"): inner-product
// scores of every query against every indexed unit vector, by matrix products over the
// embedding matrix, then partial top-k selection (Section 4.4).
//
// One launch does the whole search.  The grid is (row chunk) x (query block).  Each
// workgroup streams its chunk of rows tile by tile, scores a tile against its query block
// with MFMA (bf16 / fp16 storage, fp32 accumulation) or VALU FMA (fp32 storage), keeps a
// per-query top-k across its tiles, and appends that local top-k to a per-query candidate
// list in the workspace, skipping entries below the best k-th score any workgroup has
// published for the query (a valid lower bound of the true k-th score).  The last workgroup
// of each query block to finish merges the candidates into the final (score desc, id asc)
// list and resets the control block it used.  The score matrix never leaves the chip.
//
// Data movement for bf16 / fp16: each stage of KC = 64 dimensions is copied straight from
// global memory into an LDS ring slot with global_load_lds_dwordx4 (no VGPR round trip).
// Every wave loads its own row fragments already in MFMA lane order, so fragment reads are
// linear and conflict-free; query fragments are loaded the same way once per stage for the
// whole workgroup.  R - 1 stages stay in flight while one is consumed.
#include <algorithm>

#include "oprag_internal.h"
#include "select.h"

namespace oprag {
namespace {

using namespace dev;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

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

// Workgroup barrier without the vmcnt drain a full __syncthreads() fence would add: LDS
// traffic of this wave is complete, in-flight ring loads stay in flight.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Full barrier: every wave's global and LDS traffic is complete.
__device__ __forceinline__ void full_barrier() {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

constexpr int kThreads = 256;
constexpr int kWaves = 4;

// Logical workgroup index with consecutive indices kept on one XCD (the hardware deals
// workgroups round-robin over the 8 XCDs), so the query blocks of one row chunk share an L2.
__device__ __forceinline__ long long logical_block() {
  long long g = blockIdx.x, G = gridDim.x;
  return (G % 8 == 0) ? (g % 8) * (G / 8) + g / 8 : g;
}

// ------------------------------------------------------------------------------------
// Selection state, one of two strategies:
//   SEL 0: every thread keeps a register top-KS list for one query over a slice of the
//          tile rows (k <= KS <= 16);
//   SEL 1: every wave keeps a 128-entry sorted queue per query it owns and merges
//          batches of 64 candidates with a bitonic network (k <= 128).
// ------------------------------------------------------------------------------------
template <int BN, int KS, int SEL>
struct Selector;

template <int BN, int KS>
struct Selector<BN, KS, 0> {
  static constexpr int TPQ = kThreads / BN;  // threads per query
  static constexpr int SSTR = BN + 4;        // floats per score-tile row
  RegTopK<KS> list;

  __device__ __forceinline__ void init() { list.clear(); }

  // Scan rows [0, rows) of the LDS score tile S[row][query]; global row id = row0 + r.
  __device__ __forceinline__ void scan(const float* S, int rows, long long row0, long long row_lim, int q_lim) {
    const int t = threadIdx.x, qq = t % BN, sub = t / BN;
    if (qq >= q_lim) return;
    const int per = rows / TPQ;
    float fl = list.floor_score();
    for (int i = 0; i < per; ++i) {
      const int r = sub * per + i;
      if (row0 + r >= row_lim) break;
      const float s = S[r * SSTR + qq];
      if (s >= fl) {
        list.insert(composite(s, (uint32_t)(row0 + r)));
        fl = list.floor_score();
      }
    }
  }

  // Combine the TPQ lists of each query into the thread with sub == 0.
  __device__ __forceinline__ void combine(u64* buf) {
    const int t = threadIdx.x;
#pragma unroll
    for (int i = 0; i < KS; ++i) buf[i * kThreads + t] = list.v[i];
    lds_barrier();
    if (t < BN) {
      for (int j = 1; j < TPQ; ++j)
#pragma unroll
        for (int i = 0; i < KS; ++i) list.insert(buf[i * kThreads + t + j * BN]);
    }
    lds_barrier();
  }

  // Append this workgroup's top-k of query q (thread t < BN only).
  __device__ __forceinline__ void emit(const DenseArgs& a, int q) {
    const uint32_t gthr = __hip_atomic_load(&a.thr[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int n = 0;
    u64 kth = 0;
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      if (i < a.k && list.v[i] != 0ull && comp_key(list.v[i]) >= gthr) n = i + 1;
      if (i == a.k - 1) kth = list.v[i];
    }
    if (n) {
      const uint32_t base = atomicAdd(&a.cnt[q], (uint32_t)n);
      u64* dst = a.cand + (long long)q * a.cap + base;
#pragma unroll
      for (int i = 0; i < KS; ++i)
        if (i < n) dst[i] = list.v[i];
    }
    if (kth) atomicMax(&a.thr[q], comp_key(kth));
  }

  // Last workgroup: merge the candidates of every query of the block, write the output.
  __device__ __forceinline__ void merge_and_write(const DenseArgs& a, int q0, u64* buf) {
    const int t = threadIdx.x, qq = t % BN, sub = t / BN, q = q0 + qq;
    list.clear();
    if (q < a.nq) {
      const uint32_t nc = __hip_atomic_load(&a.cnt[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const u64* src = a.cand + (long long)q * a.cap;
      for (uint32_t j = sub; j < nc; j += TPQ) list.insert(src[j]);
    }
    combine(buf);
    if (t < BN && q < a.nq) {
#pragma unroll
      for (int i = 0; i < KS; ++i) {
        if (i < a.k) {
          const u64 c = list.v[i];
          a.out_ids[(long long)q * a.k + i] = c ? (long long)comp_row(c) : -1ll;
          a.out_scores[(long long)q * a.k + i] = c ? comp_score(c) : -__builtin_inff();
        }
      }
      a.cnt[q] = 0u;
      a.thr[q] = 0u;
    }
  }
};

template <int BN, int KS>
struct Selector<BN, KS, 1> {
  static constexpr int QPW = BN / kWaves;  // queries per wave
  static constexpr int SSTR = BN + 1;
  u64 q0[QPW], q1[QPW];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int j = 0; j < QPW; ++j) q0[j] = q1[j] = 0ull;
  }

  __device__ __forceinline__ void scan(const float* S, int rows, long long row0, long long row_lim, int q_lim) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < QPW; ++j) {
      const int qq = w + kWaves * j;
      if (qq >= q_lim) continue;
      for (int base = 0; base < rows; base += 64) {
        const int r = base + lane;
        const long long row = row0 + r;
        u64 c = 0ull;
        if (r < rows && row < row_lim) c = composite(S[r * SSTR + qq], (uint32_t)row);
        const u64 kth = queue_at(q0[j], q1[j], kk_ - 1);
        wave_offer(q0[j], q1[j], c, kth, lane);
      }
    }
  }

  __device__ __forceinline__ void combine(u64*) {}

  __device__ __forceinline__ void emit_all(const DenseArgs& a, int qbase) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < QPW; ++j) {
      const int q = qbase + w + kWaves * j;
      if (q >= a.nq) continue;
      const uint32_t gthr = __hip_atomic_load(&a.thr[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const bool v0 = lane < a.k && q0[j] != 0ull && comp_key(q0[j]) >= gthr;
      const bool v1 = lane + 64 < a.k && q1[j] != 0ull && comp_key(q1[j]) >= gthr;
      const int n0 = __popcll(__ballot(v0)), n1 = __popcll(__ballot(v1));
      const int n = n0 + n1;
      const u64 kth = queue_at(q0[j], q1[j], a.k - 1);
      if (n) {
        uint32_t base = 0;
        if (lane == 0) base = atomicAdd(&a.cnt[q], (uint32_t)n);
        base = (uint32_t)__shfl((int)base, 0, 64);
        u64* dst = a.cand + (long long)q * a.cap + base;
        if (v0) dst[lane] = q0[j];
        if (v1) dst[lane + 64] = q1[j];
      }
      if (lane == 0 && kth) atomicMax(&a.thr[q], comp_key(kth));
    }
  }

  __device__ __forceinline__ void merge_and_write(const DenseArgs& a, int qbase) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    init();
#pragma unroll
    for (int j = 0; j < QPW; ++j) {
      const int q = qbase + w + kWaves * j;
      if (q >= a.nq) continue;
      const uint32_t nc = __hip_atomic_load(&a.cnt[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const u64* src = a.cand + (long long)q * a.cap;
      for (uint32_t base = 0; base < nc; base += 64) {
        const u64 c = (base + lane < nc) ? src[base + lane] : 0ull;
        wave_offer(q0[j], q1[j], c, queue_at(q0[j], q1[j], a.k - 1), lane);
      }
      const long long o = (long long)q * a.k;
      if (lane < a.k) {
        a.out_ids[o + lane] = q0[j] ? (long long)comp_row(q0[j]) : -1ll;
        a.out_scores[o + lane] = q0[j] ? comp_score(q0[j]) : -__builtin_inff();
      }
      if (lane + 64 < a.k) {
        a.out_ids[o + lane + 64] = q1[j] ? (long long)comp_row(q1[j]) : -1ll;
        a.out_scores[o + lane + 64] = q1[j] ? comp_score(q1[j]) : -__builtin_inff();
      }
      if (lane == 0) {
        a.cnt[q] = 0u;
        a.thr[q] = 0u;
      }
    }
  }

  int kk_ = 1;  // k of the search (entry kk_ - 1 of a queue is the pruning threshold)
};

// Common tail: emission, last-workgroup detection, merge, control-block reset.
template <int BN, int KS, int SEL>
__device__ __forceinline__ void finish(Selector<BN, KS, SEL>& sel, const DenseArgs& a, int qb, unsigned char* smem) {
  const int t = threadIdx.x;
  const int q0 = qb * BN;
  u64* buf = reinterpret_cast<u64*>(smem);
  __shared__ int s_last;
  if constexpr (SEL == 0) {
    sel.combine(buf);
    if (t < BN && q0 + t < a.nq) sel.emit(a, q0 + t);
  } else {
    sel.emit_all(a, q0);
  }
  __threadfence();
  __syncthreads();
  if (t == 0) {
    const uint32_t ticket = atomicAdd(&a.done[qb], 1u);
    s_last = (ticket == (uint32_t)(a.n_chunks - 1));
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  if constexpr (SEL == 0) {
    sel.merge_and_write(a, q0, buf);
  } else {
    sel.merge_and_write(a, q0);
  }
  if (t == 0) a.done[qb] = 0u;
}

// ------------------------------------------------------------------------------------
// bf16 / fp16 MFMA kernel.
//   BN  queries per workgroup (multiple of 16), MW 16-row subtiles per wave,
//   tile = 4 waves x MW x 16 rows; stage = 64 dimensions; R ring slots.
// ------------------------------------------------------------------------------------
template <int DT, int BN, int MW, int KS, int SEL>
__global__ __launch_bounds__(kThreads) void dense_mfma_kernel(DenseArgs a) {
  using M = Mfma<DT>;
  using V = typename M::V;
  using T = typename M::T;
  constexpr int KC = 64, NS = KC / 32, R = 3;
  constexpr int NI = BN / 16;
  constexpr int TR = kWaves * MW * 16;
  constexpr int XFR = MW * NS;                 // row fragments per wave per stage
  constexpr int QFR = NI * NS;                 // query fragments per stage
  constexpr int NQF = (QFR + kWaves - 1) / kWaves;
  constexpr int NDMA = XFR + NQF;              // DMA instructions per wave per stage
  constexpr int SLOT = (kWaves * XFR + QFR) * 1024;
  using Sel = Selector<BN, KS, SEL>;
  constexpr int SSTR = Sel::SSTR;
  constexpr int SBYTES = (TR / 2) * SSTR * 4;
  constexpr int CBYTES = SEL == 0 ? KS * kThreads * 8 : 0;
  constexpr int A1 = R * SLOT > SBYTES ? R * SLOT : SBYTES;
  constexpr int SMEM = A1 > CBYTES ? A1 : CBYTES;
  static_assert(NDMA * (R - 2) < 64, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[SMEM];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const long long L = logical_block();
  const int qb = (int)(L % a.n_qblocks);
  const long long chunk = L / a.n_qblocks;
  const int q0 = qb * BN;
  const int q_lim = min(BN, a.nq - q0);
  const long long row_begin = chunk * a.rows_per_chunk;
  const long long row_end = min(row_begin + a.rows_per_chunk, a.n_rows);
  const int d = a.d;
  const int nk = d / KC;
  const T* X = static_cast<const T*>(a.X);
  const T* Q = static_cast<const T*>(a.Q);

  Sel sel;
  sel.init();
  if constexpr (SEL == 1) sel.kk_ = a.k;

  // Per-lane source offsets inside a stage (dimension offset of this lane's 8 values).
  const int kl = (lane >> 4) * 8;
  // Query fragment sources of this wave (clamped to a valid query).
  const T* qsrc[NQF];
  int qdst[NQF];
#pragma unroll
  for (int j = 0; j < NQF; ++j) {
    const int f = (w + kWaves * j) % QFR;      // waves beyond QFR repeat a fragment
    const int ni = f / NS, s = f % NS;
    const int qrow = min(q0 + ni * 16 + (lane & 15), a.nq - 1);
    qsrc[j] = Q + (long long)qrow * d + s * 32 + kl;
    qdst[j] = (kWaves * XFR + f) * 1024;
  }

  for (long long tile0 = row_begin; tile0 < row_end; tile0 += TR) {
    // Row sources of this wave for the tile (clamped to the last valid row).
    const T* xsrc[MW];
#pragma unroll
    for (int mi = 0; mi < MW; ++mi) {
      const long long row = min(tile0 + w * MW * 16 + mi * 16 + (lane & 15), a.n_rows - 1);
      xsrc[mi] = X + row * d + kl;
    }
    auto issue = [&](int c) {
      unsigned char* slot = smem + (c % R) * SLOT;
      const int kc = c * KC;
#pragma unroll
      for (int mi = 0; mi < MW; ++mi)
#pragma unroll
        for (int s = 0; s < NS; ++s)
          dma16(xsrc[mi] + kc + s * 32, slot + (w * XFR + mi * NS + s) * 1024);
#pragma unroll
      for (int j = 0; j < NQF; ++j) dma16(qsrc[j] + kc, slot + qdst[j]);
    };

    f32x4 acc[MW][NI];
#pragma unroll
    for (int mi = 0; mi < MW; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int c = 0; c < R - 1; ++c)
      if (c < nk) issue(c);

    for (int c = 0; c < nk; ++c) {
      if (c + R - 2 < nk) wait_vm<NDMA * (R - 2)>();
      else wait_vm<0>();
      lds_barrier();
      if (c + R - 1 < nk) issue(c + R - 1);
      const unsigned char* slot = smem + (c % R) * SLOT;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        V xa[MW];
#pragma unroll
        for (int mi = 0; mi < MW; ++mi)
          xa[mi] = *reinterpret_cast<const V*>(slot + (w * XFR + mi * NS + s) * 1024 + lane * 16);
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
          const V qv = *reinterpret_cast<const V*>(slot + (kWaves * XFR + ni * NS + s) * 1024 + lane * 16);
#pragma unroll
          for (int mi = 0; mi < MW; ++mi) acc[mi][ni] = M::run(xa[mi], qv, acc[mi][ni]);
        }
      }
    }
    full_barrier();

    // Epilogue: two halves of TR/2 rows through the LDS score tile (aliases the ring).
    float* S = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if ((w >> 1) == h) {
        const int rbase = (w & 1) * MW * 16;
#pragma unroll
        for (int mi = 0; mi < MW; ++mi)
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              S[(rbase + mi * 16 + (lane >> 4) * 4 + r) * SSTR + ni * 16 + (lane & 15)] = acc[mi][ni][r];
      }
      lds_barrier();
      sel.scan(S, TR / 2, tile0 + h * (TR / 2), row_end, q_lim);
      lds_barrier();
    }
  }
  finish(sel, a, qb, smem);
}

// ------------------------------------------------------------------------------------
// fp32 VALU kernel: tile of 64 rows x BN = 32 queries, 32 dimensions per stage.
// ------------------------------------------------------------------------------------
template <int KS, int SEL>
__global__ __launch_bounds__(kThreads) void dense_f32_kernel(DenseArgs a) {
  constexpr int BN = 32, TR = 64, KC = 32;
  using Sel = Selector<BN, KS, SEL>;
  constexpr int SSTR = Sel::SSTR;
  constexpr int XB = TR * (KC + 1) * 4, QB = BN * (KC + 1) * 4, SB = TR * SSTR * 4;
  constexpr int CB = SEL == 0 ? KS * kThreads * 8 : 0;
  constexpr int A1 = XB + QB > SB ? XB + QB : SB;
  constexpr int SMEM = A1 > CB ? A1 : CB;
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
  if constexpr (SEL == 1) sel.kk_ = a.k;

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
    for (int r = 0; r < 8; ++r) S[(rg * 8 + r) * SSTR + qq] = acc[r];
    __syncthreads();
    sel.scan(S, TR, tile0, row_end, q_lim);
    __syncthreads();
  }
  finish(sel, a, qb, smem);
}

// ------------------------------------------------------------------------------------
// Kernel table and planning.
// ------------------------------------------------------------------------------------
struct KernelInfo {
  void (*fn)(DenseArgs);
  int dtype, bn, tile_rows, ks, sel, wgs_per_cu;
};

#define MF(DT, BN, MW, KS, SEL, OCC) \
  {dense_mfma_kernel<DT, BN, MW, KS, SEL>, DT, BN, kWaves * MW * 16, KS, SEL, OCC}

const KernelInfo kKernels[] = {
    // fp32 (VALU)
    {dense_f32_kernel<8, 0>, kDtypeF32, 32, 64, 8, 0, 2},
    {dense_f32_kernel<16, 0>, kDtypeF32, 32, 64, 16, 0, 2},
    {dense_f32_kernel<8, 1>, kDtypeF32, 32, 64, 128, 1, 2},
    // bf16
    MF(kDtypeBF16, 128, 4, 8, 0, 1), MF(kDtypeBF16, 128, 4, 16, 0, 1),
    MF(kDtypeBF16, 64, 2, 8, 0, 2), MF(kDtypeBF16, 64, 2, 16, 0, 2),
    MF(kDtypeBF16, 16, 1, 8, 0, 4), MF(kDtypeBF16, 16, 1, 16, 0, 4),
    MF(kDtypeBF16, 32, 4, 8, 1, 1),
    // fp16
    MF(kDtypeF16, 128, 4, 8, 0, 1), MF(kDtypeF16, 128, 4, 16, 0, 1),
    MF(kDtypeF16, 64, 2, 8, 0, 2), MF(kDtypeF16, 64, 2, 16, 0, 2),
    MF(kDtypeF16, 16, 1, 8, 0, 4), MF(kDtypeF16, 16, 1, 16, 0, 4),
    MF(kDtypeF16, 32, 4, 8, 1, 1),
};
constexpr int kNumKernels = sizeof(kKernels) / sizeof(kKernels[0]);

int pick_kernel(int dtype, int nq, int k) {
  const int sel = k <= 16 ? 0 : 1;
  const int ks = k <= 8 ? 8 : 16;
  int want_bn = 32;
  if (dtype != kDtypeF32 && sel == 0) want_bn = nq > 64 ? 128 : (nq > 16 ? 64 : 16);
  for (int i = 0; i < kNumKernels; ++i) {
    const KernelInfo& ki = kKernels[i];
    if (ki.dtype != dtype || ki.sel != sel || ki.bn != want_bn) continue;
    if (sel == 0 && ki.ks != ks) continue;
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
  const long long target = (long long)kNumCUs * ki.wgs_per_cu * 2;
  long long chunks = (target + p.n_qblocks - 1) / p.n_qblocks;
  if (ki.sel == 1) chunks = std::min(chunks, std::max(1ll, n_tiles / 4));
  chunks = std::max(1ll, std::min(chunks, n_tiles));
  const long long tiles_per_chunk = n_tiles ? (n_tiles + chunks - 1) / chunks : 1;
  p.rows_per_chunk = tiles_per_chunk * p.tile_rows;
  p.n_chunks = (int)std::max(1ll, n_tiles ? (n_tiles + tiles_per_chunk - 1) / tiles_per_chunk : 1);
  p.cap = (long long)p.n_chunks * k;
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
  return hipLaunchKernel(reinterpret_cast<const void*>(ki.fn), dim3((unsigned)p.grid), dim3(kThreads), params, 0, s);
}

}  // namespace oprag
