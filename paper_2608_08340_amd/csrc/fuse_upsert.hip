// Reciprocal rank fusion of a dense and a sparse top list, and append-only upsert.
//
// Fusion: the hybrid path combines dense and lexical evidence over the full corpus
// (Section 4.4).  The hybrid workload fuses the two top lists with reciprocal rank fusion
// (Cormack, Clarke and Buettcher, SIGIR 2009): fused(d) = sum over the lists L holding d of
// 1 / (k_rrf + rank_L(d)), 1-based ranks.  Fused values are compared exactly as fractions
// num / den in 64-bit integers (den = product of at most two (k_rrf + rank) factors), so
// exact ties such as 1/63 = 2/126 stay ties and are broken by ascending id.
//
// Upsert: Op_upsert (Section 3.2, "Upsert") inserts new embeddings, I' = Op_upsert(I, E; b_u),
// committed in bulk.  Here: rows are appended at ids n_rows .. n_rows + m - 1 of a
// preallocated slab, converting fp32 input to the slab's bf16 / fp16 with
// round-to-nearest-even when the dtypes differ.
#include <algorithm>

#include "oprag_internal.h"
#include "select.h"

namespace oprag {
namespace {

using namespace dev;

constexpr int kMaxCand = 2 * kMaxK;

// One workgroup of 256 threads per query: thread t < kd owns dense entry t, thread kd + j owns
// sparse entry j (kd, ks <= 128).  Both lists are staged in LDS; every candidate's rank is the
// number of candidates that beat it in the exact rational order (fused desc, id asc), and a
// thread stops counting once its candidate is out of the first k.
constexpr int kRrfThreads = 256;
__global__ __launch_bounds__(kRrfThreads) void rrf_kernel(const long long* dense_ids, int kd,
                                                          const long long* sparse_ids, int ks, long long nq, int rrf_k,
                                                          int k, float* out_fused, long long* out_ids) {
  __shared__ long long dn_ids[kMaxK];
  __shared__ long long sp_ids[kMaxK];
  __shared__ long long cid[kMaxCand];
  __shared__ long long cnum[kMaxCand];
  __shared__ long long cden[kMaxCand];
  __shared__ double cval[kMaxCand];
  __shared__ int s_nc;
  const long long q = blockIdx.x;
  const int t = threadIdx.x;
  const long long* D = dense_ids + q * kd;
  const long long* S = sparse_ids + q * ks;
  if (t < kd) dn_ids[t] = D[t];
  if (t < ks) sp_ids[t] = S[t];
  if (t == 0) s_nc = 0;
  __syncthreads();
  long long id = -1, num = 0, den = 1;
  if (t < kd) {  // dense entry: rank t + 1, plus its sparse rank when present
    id = dn_ids[t];
    if (id >= 0) {
      const long long a = (long long)rrf_k + t + 1;
      num = 1;
      den = a;
      int hit = -1;
      for (int j = 0; j < ks; j += 8) {  // eight independent LDS reads per step
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (j + u < ks && hit < 0 && sp_ids[j + u] == id) hit = j + u;
        if (hit >= 0) break;
      }
      if (hit >= 0) {
        const long long b = (long long)rrf_k + hit + 1;
        num = a + b;
        den = a * b;
      }
    }
  } else if (t - kd < ks) {  // sparse entry absent from the dense list
    const int j = t - kd;
    id = sp_ids[j];
    if (id >= 0) {
      bool dup = false;
      for (int i = 0; i < kd && !dup; i += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u) dup |= i + u < kd && dn_ids[i + u] == id;
      }
      if (dup) id = -1;
      num = 1;
      den = (long long)rrf_k + j + 1;
    }
  }
  if (id >= 0) {
    const int slot = atomicAdd(&s_nc, 1);
    cid[slot] = id;
    cnum[slot] = num;
    cden[slot] = den;
    cval[slot] = (double)num / (double)den;
  }
  __syncthreads();
  const int nc = s_nc;
  if (t < nc) {
    // Rank = candidates that beat this one.  The correctly rounded quotients order any two
    // fused values that differ by more than a few ulps; closer pairs (exact ties such as
    // 1/63 = 2/126 among them) are compared exactly as int64 cross products.
    const long long n0 = cnum[t], d0 = cden[t], id0 = cid[t];
    const double v0 = cval[t], hi = v0 * (1.0 + 1e-14), lo = v0 * (1.0 - 1e-14);
    int rank = 0;
    for (int o = 0; o < nc && rank < k; o += 8) {  // eight candidates per step
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (o + u < nc) {
          const double v = cval[o + u];
          bool beats = v > hi;
          if (!beats && v >= lo) {
            const long long lhs = cnum[o + u] * d0, rhs = n0 * cden[o + u];
            beats = lhs > rhs || (lhs == rhs && cid[o + u] < id0);
          }
          rank += beats ? 1 : 0;
        }
      }
    }
    if (rank < k) {
      out_ids[q * k + rank] = id0;
      out_fused[q * k + rank] = (float)((double)n0 / (double)d0);
    }
  }
  for (int r = nc + t; r < k; r += kRrfThreads) {
    out_ids[q * k + r] = -1;
    out_fused[q * k + r] = -__builtin_inff();
  }
}

__device__ __forceinline__ unsigned short f32_to_bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (unsigned short)((u >> 16) | 0x40u);  // NaN stays (quiet) NaN
  return (unsigned short)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// Same-dtype copy, 16 bytes per thread per step.
__global__ void copy16_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, long long n16) {
  const long long stride = (long long)gridDim.x * blockDim.x;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) dst[i] = src[i];
}

// fp32 -> bf16 (DT 1) or fp16 (DT 2), 8 elements per thread per step.
template <int DT>
__global__ void convert8_kernel(const float4* __restrict__ src, uint4* __restrict__ dst, long long n8) {
  const long long stride = (long long)gridDim.x * blockDim.x;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += stride) {
    const float4 a = src[2 * i], b = src[2 * i + 1];
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    unsigned short h[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if constexpr (DT == kDtypeBF16) {
        h[j] = f32_to_bf16_rne(v[j]);
      } else {
        _Float16 f = (_Float16)v[j];  // v_cvt_f16_f32: round to nearest even
        h[j] = __builtin_bit_cast(unsigned short, f);
      }
    }
    uint4 o;
    o.x = h[0] | ((uint32_t)h[1] << 16);
    o.y = h[2] | ((uint32_t)h[3] << 16);
    o.z = h[4] | ((uint32_t)h[5] << 16);
    o.w = h[6] | ((uint32_t)h[7] << 16);
    dst[i] = o;
  }
}

}  // namespace

hipError_t launch_rrf(const long long* dense_ids, int k_dense, const long long* sparse_ids, int k_sparse, long long nq,
                      int rrf_k, int k, float* out_fused, long long* out_ids, hipStream_t s) {
  hipLaunchKernelGGL(rrf_kernel, dim3((unsigned)nq), dim3(kRrfThreads), 0, s, dense_ids, k_dense, sparse_ids, k_sparse,
                     nq, rrf_k, k, out_fused, out_ids);
  return hipGetLastError();
}

hipError_t launch_upsert(void* slab, int slab_dtype, int d, long long first_row, const void* rows, int rows_dtype,
                         long long m, hipStream_t s) {
  const size_t es = slab_dtype == kDtypeF32 ? 4 : 2;
  unsigned char* dst = static_cast<unsigned char*>(slab) + (size_t)first_row * d * es;
  const long long n = m * (long long)d;
  if (rows_dtype == slab_dtype) {
    const long long n16 = n * (long long)es / 16;
    const int blocks = (int)std::min<long long>(4096, (n16 + 255) / 256);
    hipLaunchKernelGGL(copy16_kernel, dim3(std::max(1, blocks)), dim3(256), 0, s, static_cast<const uint4*>(rows),
                       reinterpret_cast<uint4*>(dst), n16);
  } else {
    const long long n8 = n / 8;
    const int blocks = (int)std::min<long long>(4096, (n8 + 255) / 256);
    if (slab_dtype == kDtypeBF16)
      hipLaunchKernelGGL(convert8_kernel<kDtypeBF16>, dim3(std::max(1, blocks)), dim3(256), 0, s,
                         static_cast<const float4*>(rows), reinterpret_cast<uint4*>(dst), n8);
    else
      hipLaunchKernelGGL(convert8_kernel<kDtypeF16>, dim3(std::max(1, blocks)), dim3(256), 0, s,
                         static_cast<const float4*>(rows), reinterpret_cast<uint4*>(dst), n8);
  }
  return hipGetLastError();
}

}  // namespace oprag
