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
#include "rrf.h"
#include "select.h"

namespace oprag {
namespace {

using namespace dev;

// One workgroup of 256 threads per query (rrf_query in rrf.h).
constexpr int kRrfThreads = 256;
__global__ __launch_bounds__(kRrfThreads) void rrf_kernel(const long long* dense_ids, int kd,
                                                          const long long* sparse_ids, int ks, long long nq, int rrf_k,
                                                          int k, float* out_fused, long long* out_ids) {
  __shared__ __attribute__((aligned(16))) unsigned char area[RrfScratch::kBytes];
  const long long q = blockIdx.x;
  rrf_query<kRrfThreads>(dense_ids + q * kd, kd, sparse_ids + q * ks, ks, rrf_k, k, out_fused + q * k, out_ids + q * k,
                         RrfScratch(area));
}

constexpr int kMaxPoolDim = 8192;  // OPRAG_MAX_DIM

__device__ __forceinline__ unsigned short f32_to_bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (unsigned short)((u >> 16) | 0x40u);  // NaN stays (quiet) NaN
  return (unsigned short)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// Read-bandwidth probe (diagnostics): a plain streaming read of n16 16-byte words, eight
// loads in flight per thread, grid-strided; each workgroup folds what it read into one word
// (so the loads cannot be dropped) and writes it to sink[blockIdx.x].
__global__ __launch_bounds__(256) void probe_read_kernel(const uint4* __restrict__ src, long long n16,
                                                        unsigned int* __restrict__ sink) {
  __shared__ unsigned int part[4];
  const long long stride = (long long)gridDim.x * 256 * 8;
  unsigned int x = 0u;
  for (long long i0 = (long long)blockIdx.x * 256 * 8 + threadIdx.x; i0 < n16; i0 += stride) {
    uint4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = i0 + u * 256 < n16 ? src[i0 + u * 256] : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int u = 0; u < 8; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x ^= (unsigned int)__shfl_xor((int)x, o);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
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

// Embedding tail fused with the upsert (Section 4.3: mean pool over the chunk's tokens, then L2
// normalisation; Section 3.2: Op_upsert).  One workgroup of 1,024 threads per chunk.  Thread t
// owns eight consecutive dimensions 8 (t % 128) + 1024 b of every block b and the tokens
// congruent to p = t / 128 modulo 8: it sums them in fp32 (16-byte loads of eight dimensions,
// four tokens in flight), the eight partial sums are added through LDS in the order p = 0 .. 7,
// and the squares of the sums are added in fp64.  The chunk's vector is sum / ||sum|| (the mean's 1/len cancels), rounded to
// the slab dtype, or 0 when len = 0 or the sum is 0.  len is clamped to [0, T].
constexpr int kPoolThreads = 1024;
constexpr int kPoolLanes = 128;                         // threads per token residue
constexpr int kPoolPar = kPoolThreads / kPoolLanes;     // token residues (8)
template <int HT>
__device__ __forceinline__ void load8(const void* p, long long idx, int valid, float (&v)[8]) {
  if constexpr (HT == kDtypeF32) {
    const float* f = static_cast<const float*>(p) + idx;
    if (valid == 8) {
      const float4 a = *reinterpret_cast<const float4*>(f), b = *reinterpret_cast<const float4*>(f + 4);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = e < valid ? f[e] : 0.f;
    }
  } else {
    const unsigned short* h = static_cast<const unsigned short*>(p) + idx;
    if (valid == 8) {
      const uint4 a = *reinterpret_cast<const uint4*>(h);
      const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] = __uint_as_float(w[e] << 16);  // bf16 -> fp32 is exact
        v[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = e < valid ? __uint_as_float((uint32_t)h[e] << 16) : 0.f;
    }
  }
}

template <int HT, int DT>
__global__ __launch_bounds__(kPoolThreads) void pool_upsert_kernel(const void* __restrict__ hidden,
                                                                   const int* __restrict__ lengths, int T, int h,
                                                                   void* __restrict__ rows) {
  __shared__ float sums[kMaxPoolDim];
  __shared__ float part[kPoolPar - 1][kPoolLanes * 8];
  __shared__ double red[kPoolThreads / 64];
  const long long i = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int c = t % kPoolLanes, par = t / kPoolLanes;
  const int len = min(max(lengths[i], 0), T);
  const bool vec = (h & 7) == 0;  // 16-byte aligned eight-dimension pieces
  double sq = 0.0;
  const int n_blk = (h + 8 * kPoolLanes - 1) / (8 * kPoolLanes);  // the same for every thread
  for (int blk = 0; blk < n_blk; ++blk) {
    const int d0 = blk * 8 * kPoolLanes + 8 * c;
    const int valid = d0 >= h ? 0 : (vec ? 8 : min(8, h - d0));
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int tok = valid > 0 ? par : len;  // a thread past the last dimension sums nothing
    for (; tok + 3 * kPoolPar < len; tok += 4 * kPoolPar) {  // four tokens, kPoolPar apart
      float v[4][8];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        load8<HT>(hidden, ((i * T) + tok + kPoolPar * u) * (long long)h + d0, valid, v[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) s[e] += v[u][e];
    }
    for (; tok < len; tok += kPoolPar) {
      float v[8];
      load8<HT>(hidden, ((i * T) + tok) * (long long)h + d0, valid, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] += v[e];
    }
    if (par > 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) part[par - 1][c * 8 + e] = s[e];
    }
    __syncthreads();
    if (par == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float x = s[e];
#pragma unroll
        for (int u = 0; u < kPoolPar - 1; ++u) x += part[u][c * 8 + e];
        if (e < valid) {
          sums[d0 + e] = x;
          sq += (double)x * (double)x;
        }
      }
    }
    __syncthreads();  // part is rewritten by the next block
  }
  for (int o = 32; o > 0; o >>= 1) sq += __shfl_xor(sq, o);
  if (lane == 0) red[w] = sq;
  __syncthreads();
  double tot = 0.0;
#pragma unroll
  for (int u = 0; u < kPoolThreads / 64; ++u) tot += red[u];
  const double inv = tot > 0.0 ? 1.0 / sqrt(tot) : 0.0;
  for (int d = t; d < h; d += kPoolThreads) {
    const float x = (float)((double)sums[d] * inv);
    if constexpr (DT == kDtypeF32) {
      static_cast<float*>(rows)[i * h + d] = x;
    } else if constexpr (DT == kDtypeBF16) {
      static_cast<unsigned short*>(rows)[i * h + d] = f32_to_bf16_rne(x);
    } else {
      const _Float16 f = (_Float16)x;  // v_cvt_f16_f32: round to nearest even
      static_cast<unsigned short*>(rows)[i * h + d] = __builtin_bit_cast(unsigned short, f);
    }
  }
}

}  // namespace

hipError_t launch_pool_upsert(void* slab, int slab_dtype, int d, long long first_row, const void* hidden,
                              int hidden_dtype, const int* lengths, long long m, int T, hipStream_t s) {
  if (d > kMaxPoolDim) return hipErrorInvalidValue;
  const size_t es = slab_dtype == kDtypeF32 ? 4 : 2;
  void* dst = static_cast<unsigned char*>(slab) + (size_t)first_row * d * es;
  const dim3 g((unsigned)m), b(kPoolThreads);
#define OPRAG_POOL(HT, DT) hipLaunchKernelGGL((pool_upsert_kernel<HT, DT>), g, b, 0, s, hidden, lengths, T, d, dst)
  if (hidden_dtype == kDtypeBF16) {
    if (slab_dtype == kDtypeBF16) OPRAG_POOL(kDtypeBF16, kDtypeBF16);
    else if (slab_dtype == kDtypeF16) OPRAG_POOL(kDtypeBF16, kDtypeF16);
    else OPRAG_POOL(kDtypeBF16, kDtypeF32);
  } else {
    if (slab_dtype == kDtypeBF16) OPRAG_POOL(kDtypeF32, kDtypeBF16);
    else if (slab_dtype == kDtypeF16) OPRAG_POOL(kDtypeF32, kDtypeF16);
    else OPRAG_POOL(kDtypeF32, kDtypeF32);
  }
#undef OPRAG_POOL
  return hipGetLastError();
}

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

hipError_t launch_probe_read(const void* src, long long bytes, unsigned int* sink, int blocks, hipStream_t s) {
  hipLaunchKernelGGL(probe_read_kernel, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<const uint4*>(src),
                     bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace oprag
