// Device-side top-k selection primitives shared by the dense and sparse kernels.
//
// Partial top-k selection instead of a full sort is one of the three exact retrieval
// optimisations the paper credits for its hybrid-retrieval speed-up (Section 4.4; Section 5.5).
// Order used everywhere: score descending, then row id ascending.  A (score, row) pair is
// packed into one 64-bit "composite" whose unsigned order is exactly that order, so every
// comparison below is a single 64-bit compare.  Composite 0 is the empty slot (it sorts
// below every finite score).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace oprag {
namespace dev {

typedef unsigned long long u64;

// fp32 -> order-preserving unsigned key; -0 and +0 share a key.
__device__ __forceinline__ uint32_t score_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u << 1) == 0u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_score(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

__device__ __forceinline__ u64 composite(float s, uint32_t row) {
  return ((u64)score_key(s) << 32) | (u64)(uint32_t)(~row);
}
__device__ __forceinline__ uint32_t comp_row(u64 c) { return ~(uint32_t)c; }
__device__ __forceinline__ float comp_score(u64 c) { return key_score((uint32_t)(c >> 32)); }
__device__ __forceinline__ uint32_t comp_key(u64 c) { return (uint32_t)(c >> 32); }
__device__ __forceinline__ u64 umax64(u64 a, u64 b) { return a > b ? a : b; }
__device__ __forceinline__ u64 umin64(u64 a, u64 b) { return a < b ? a : b; }

// Per-thread sorted (descending) list of the KS best composites seen so far.
template <int KS>
struct RegTopK {
  u64 v[KS];
  __device__ __forceinline__ void clear() {
#pragma unroll
    for (int i = 0; i < KS; ++i) v[i] = 0ull;
  }
  // Top-KS of v + {x}: new[i] = max(v[i], min(v[i-1], x)), new[0] = max(v[0], x).
  __device__ __forceinline__ void insert(u64 x) {
#pragma unroll
    for (int i = KS - 1; i > 0; --i) v[i] = umax64(v[i], umin64(v[i - 1], x));
    v[0] = umax64(v[0], x);
  }
  // Lowest score that could still enter the list (-inf while it is not full).
  __device__ __forceinline__ float floor_score() const {
    return v[KS - 1] ? comp_score(v[KS - 1]) : -__builtin_inff();
  }
};

// ------------------------------------------------------------------ wave64 bitonic network

__device__ __forceinline__ u64 shfl_xor64(u64 x, int m) {
  int lo = __shfl_xor((int)(uint32_t)x, m, 64);
  int hi = __shfl_xor((int)(uint32_t)(x >> 32), m, 64);
  return ((u64)(uint32_t)hi << 32) | (u64)(uint32_t)lo;
}

__device__ __forceinline__ u64 readlane64(u64 x, int lane) {
  uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, lane);
  uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), lane);
  return ((u64)hi << 32) | lo;
}

// Sort one value per lane across the 64 lanes, descending by lane index.
__device__ __forceinline__ u64 wave_sort64_desc(u64 x, int lane) {
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1) {
#pragma unroll
    for (int j = size >> 1; j > 0; j >>= 1) {
      u64 y = shfl_xor64(x, j);
      bool lower = (lane & j) == 0;
      bool desc = (lane & size) == 0;
      x = (lower == desc) ? umax64(x, y) : umin64(x, y);
    }
  }
  return x;
}

// Queue of 128 composites sorted descending: entry i in lane i of q0, entry 64+i in lane i
// of q1.  Merges 64 candidates (sorted descending across lanes) and keeps the best 128.
// Max of a descending sequence and a reversed (ascending) one yields the best half of the
// union as a bitonic sequence, which the half-cleaner cascade then sorts.
__device__ __forceinline__ void wave_merge128(u64& q0, u64& q1, u64 c_sorted, int lane) {
  u64 t = umax64(q1, shfl_xor64(c_sorted, 63));
  u64 a = umax64(q0, t), b = umin64(q0, t);
#pragma unroll
  for (int j = 32; j > 0; j >>= 1) {
    u64 ya = shfl_xor64(a, j), yb = shfl_xor64(b, j);
    bool lower = (lane & j) == 0;
    a = lower ? umax64(a, ya) : umin64(a, ya);
    b = lower ? umax64(b, yb) : umin64(b, yb);
  }
  q0 = a;
  q1 = b;
}

// Entry i (0 <= i < 128, wave-uniform) of a 128-queue.
__device__ __forceinline__ u64 queue_at(u64 q0, u64 q1, int i) {
  return i < 64 ? readlane64(q0, i) : readlane64(q1, i - 64);
}

// Offer one candidate per lane (0 = none) to a 128-queue; keeps the best 128.
__device__ __forceinline__ void wave_offer(u64& q0, u64& q1, u64 c, u64 kth, int lane) {
  bool take = c > kth;
  if (__ballot(take)) {
    c = take ? c : 0ull;
    wave_merge128(q0, q1, wave_sort64_desc(c, lane), lane);
  }
}

// Weighted fusion of one chunk: sd (x - mnd) + sl (y - mnl) in fp64 with every operation
// rounded explicitly, then rounded to fp32 (sd = w_d / (max_d - min_d), 0 for a constant row;
// likewise sl), so every kernel that fuses gives the same value.
__device__ __forceinline__ float fused_value(double sd, double sl, double mnd, double mnl, float x, float y) {
  const double v = __dadd_rn(__dmul_rn(sd, __dsub_rn((double)x, mnd)), __dmul_rn(sl, __dsub_rn((double)y, mnl)));
  return __double2float_rn(v);
}

}  // namespace dev
}  // namespace oprag
