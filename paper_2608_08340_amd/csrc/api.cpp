// Host runtime behind the C ABI of include/oprag.h: argument validation (always complete
// before the first HIP call), the index handle, workspace planning and kernel dispatch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/oprag.h"
#include "oprag_internal.h"

using oprag::kMaxK;
using oprag::kMaxQPerLaunch;

struct oprag_index {
  int32_t dim = 0, dtype = 0, device = 0;
  int32_t n_cus = 0;  // compute units of the device (kernel grids are planned for it)
  int64_t capacity = 0;
  void* slab = nullptr;
  size_t slab_bytes = 0;
  int64_t n_rows = 0;
  bool has_sparse = false;
  oprag::SparseIndex sp;
  void* sp_mem = nullptr;
};

namespace {

thread_local std::string g_err;
thread_local bool t_time_armed = false;  // oprag_time_next_dense_kernel
thread_local void* t_time_ev[2] = {nullptr, nullptr};

oprag_status fail(oprag_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

oprag_status ok() {
  g_err.clear();
  return OPRAG_OK;
}

oprag_status hip_fail(hipError_t e, const char* what) {
  return fail(OPRAG_E_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

size_t elem_size(int32_t dt) { return dt == OPRAG_F32 ? 4 : 2; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool valid_dtype(int32_t dt) { return dt == OPRAG_F32 || dt == OPRAG_BF16 || dt == OPRAG_F16; }

// Makes idx->device current for the scope and restores the caller's device.
class DeviceScope {
 public:
  explicit DeviceScope(int dev) {
    err_ = hipGetDevice(&prev_);
    if (err_ == hipSuccess && prev_ != dev) {
      err_ = hipSetDevice(dev);
      switched_ = err_ == hipSuccess;
    }
  }
  ~DeviceScope() {
    if (switched_) (void)hipSetDevice(prev_);
  }
  hipError_t error() const { return err_; }

 private:
  int prev_ = 0;
  bool switched_ = false;
  hipError_t err_ = hipSuccess;
};

oprag_status check_index(const oprag_index* idx) {
  if (!idx) return fail(OPRAG_E_INVALID, "index handle is NULL");
  return OPRAG_OK;
}

oprag_status check_k(int32_t k, const char* name) {
  if (k < 1 || k > kMaxK) return fail(OPRAG_E_INVALID, "%s = %d outside [1, %d]", name, k, kMaxK);
  return OPRAG_OK;
}

oprag_status check_buf(const void* p, const char* name) {
  if (!p) return fail(OPRAG_E_INVALID, "%s is NULL", name);
  if (!aligned16(p)) return fail(OPRAG_E_INVALID, "%s is not 16-byte aligned", name);
  return OPRAG_OK;
}

size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

size_t dense_ws(const oprag_index* idx, int64_t nq, int32_t k) {
  const int nql = (int)std::min<int64_t>(nq, kMaxQPerLaunch);
  return oprag::dense_workspace_bound(idx->dtype, idx->dim, idx->capacity, nql, k, idx->n_cus);
}

size_t sparse_ws(const oprag_index* idx, int64_t nq, int32_t k) {
  return oprag::sparse_workspace_bytes(idx->has_sparse ? idx->sp.n_docs : idx->capacity, (int)nq, k);
}

size_t hybrid_ws(const oprag_index* idx, int64_t nq, int32_t kd, int32_t ks) {
  const size_t lists = align_up((size_t)nq * kd * 8) + align_up((size_t)nq * kd * 4) +
                       align_up((size_t)nq * ks * 8) + align_up((size_t)nq * ks * 4);
  return lists + std::max(align_up(dense_ws(idx, nq, kd)), align_up(sparse_ws(idx, nq, ks)));
}

// Dense-first: the candidates' ids and scores, then the dense search's own area.
size_t dense_first_ws(const oprag_index* idx, int64_t nq, int32_t n_cand) {
  return align_up((size_t)nq * n_cand * 8) + align_up((size_t)nq * n_cand * 4) + align_up(dense_ws(idx, nq, n_cand));
}

// Weighted fusion: dense scores, lexical scores (each [nq x ld], ld = capacity rounded up to
// 4), composites [nq x capacity], counts [nq].
long long weighted_ld(const oprag_index* idx) { return (idx->capacity + 3) & ~3ll; }
// Partial minima and maxima per query: of the dense dump's chunks (at most as many as its plan
// at full capacity has) and of the BM25 ranges.
int weighted_pd(const oprag_index* idx, int64_t nq) {
  return std::max(1, oprag::plan_dense_dump(idx->dtype, idx->dim, idx->capacity, (int)nq, idx->n_cus).n_chunks);
}
int weighted_pl(const oprag_index* idx) {
  return (int)((idx->capacity + oprag::kSparseRange - 1) / oprag::kSparseRange);
}
size_t weighted_ws(const oprag_index* idx, int64_t nq) {
  const size_t ld = (size_t)weighted_ld(idx);
  return 2 * align_up((size_t)nq * ld * 4) + align_up((size_t)nq * (size_t)idx->capacity * 8) + align_up((size_t)nq * 4) +
         align_up((size_t)nq * (size_t)weighted_pd(idx, nq) * 8) + align_up((size_t)nq * (size_t)weighted_pl(idx) * 8);
}

oprag_status do_dense(const oprag_index* idx, const void* q, int64_t nq, int32_t k, float* scores, int64_t* ids, void* ws,
                      size_t ws_bytes, hipStream_t s) {
  const size_t es = elem_size(idx->dtype);
  for (int64_t q0 = 0; q0 < nq; q0 += kMaxQPerLaunch) {
    const int nql = (int)std::min<int64_t>(kMaxQPerLaunch, nq - q0);
    const oprag::DensePlan p = oprag::plan_dense(idx->dtype, idx->dim, idx->n_rows, nql, k, idx->n_cus);
    if (p.kernel < 0) return fail(OPRAG_E_UNSUPPORTED, "no dense kernel for dtype %d, k %d", idx->dtype, k);
    if (oprag::dense_workspace_bytes(p, nql) > ws_bytes)
      return fail(OPRAG_E_INVALID, "workspace too small: %zu < %zu bytes", ws_bytes,
                  oprag::dense_workspace_bytes(p, nql));
    oprag::DenseArgs a;
    a.X = idx->slab;
    a.n_rows = idx->n_rows;
    a.d = idx->dim;
    a.Q = static_cast<const unsigned char*>(q) + (size_t)q0 * idx->dim * es;
    a.nq = nql;
    a.k = k;
    a.n_qblocks = p.n_qblocks;
    a.n_chunks = p.n_chunks;
    a.rows_per_chunk = p.rows_per_chunk;
    a.partial = static_cast<unsigned long long*>(ws);
    a.out_scores = scores + q0 * k;
    a.out_ids = reinterpret_cast<long long*>(ids) + q0 * k;
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    if (q0 == 0 && t_time_armed) {
      ev0 = static_cast<hipEvent_t>(t_time_ev[0]);
      ev1 = static_cast<hipEvent_t>(t_time_ev[1]);
      t_time_armed = false;
    }
    hipError_t e = oprag::launch_dense(p, idx->dtype, a, s, ev0, ev1);
    if (e != hipSuccess) return hip_fail(e, "dense search launch");
  }
  return OPRAG_OK;
}

// Largest workspace one call of a dense search without allocation may need.  The plan of
// one launch (at most kMaxQPerLaunch queries) at the current row count decides it.
size_t dense_ws_now(const oprag_index* idx, int64_t nq, int32_t k) {
  const int nql = (int)std::min<int64_t>(nq, kMaxQPerLaunch);
  const oprag::DensePlan p = oprag::plan_dense(idx->dtype, idx->dim, idx->n_rows, nql, k, idx->n_cus);
  return p.kernel < 0 ? 0 : oprag::dense_workspace_bytes(p, nql);
}

// The workspace of oprag_search_dense_noalloc: a fixed device array, one copy per GPU the
// library runs on, held until the process ends.  Host code never passes `scratch` itself to
// a kernel (on the host the name is only a stand-in for the symbol): it takes the device
// address that hipGetSymbolAddress returns, once per device, with that device current.
constexpr size_t kNoallocScratchBytes = (size_t)OPRAG_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) static unsigned char scratch[kNoallocScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch array (the device must be current).
oprag_status scratch_of(int device, void** out) {
  if (device < 0 || device >= kMaxDevices) return fail(OPRAG_E_UNSUPPORTED, "device %d >= %d", device, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(OPRAG_E_DEVICE, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[device] = p;
  }
  *out = g_scratch_ptr[device];
  return OPRAG_OK;
}

}  // namespace

extern "C" {

int32_t oprag_abi_version(void) { return OPRAG_ABI_VERSION; }

oprag_status oprag_time_next_dense_kernel(void* start_event, void* stop_event) {
  if (!start_event != !stop_event) return fail(OPRAG_E_INVALID, "pass both events or neither");
  t_time_ev[0] = start_event;
  t_time_ev[1] = stop_event;
  t_time_armed = start_event != nullptr;
  return OPRAG_OK;
}

oprag_status oprag_probe_read(const void* src_dev, size_t bytes, int32_t blocks, uint32_t* sink_dev, void* stream) {
  if (oprag_status st = check_buf(src_dev, "src_dev")) return st;
  if (oprag_status st = check_buf(sink_dev, "sink_dev")) return st;
  if (bytes == 0 || bytes % 16) return fail(OPRAG_E_INVALID, "bytes %zu is not a positive multiple of 16", bytes);
  if (blocks < 1 || blocks > OPRAG_PROBE_MAX_BLOCKS)
    return fail(OPRAG_E_INVALID, "blocks %d outside [1, %d]", blocks, OPRAG_PROBE_MAX_BLOCKS);
  const hipError_t e = oprag::launch_probe_read(src_dev, (long long)bytes, sink_dev, blocks, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "probe launch");
  return ok();
}

const char* oprag_last_error(void) { return g_err.c_str(); }

oprag_status oprag_index_create(const oprag_index_desc* desc, void* slab_dev, size_t slab_bytes, oprag_index** out) {
  if (!out) return fail(OPRAG_E_INVALID, "out is NULL");
  *out = nullptr;
  if (!desc) return fail(OPRAG_E_INVALID, "desc is NULL");
  if (!valid_dtype(desc->dtype)) return fail(OPRAG_E_INVALID, "dtype %d is not an oprag_dtype", desc->dtype);
  if (desc->dim < 1 || desc->dim > OPRAG_MAX_DIM) return fail(OPRAG_E_INVALID, "dim %d outside [1, %d]", desc->dim, OPRAG_MAX_DIM);
  if (desc->dtype == OPRAG_F32 && desc->dim % 4)
    return fail(OPRAG_E_UNSUPPORTED, "fp32 dim %d is not a multiple of 4", desc->dim);
  if (desc->dtype != OPRAG_F32 && desc->dim % 128)
    return fail(OPRAG_E_UNSUPPORTED, "bf16/fp16 dim %d is not a multiple of 128", desc->dim);
  if (desc->capacity < 1 || desc->capacity > (int64_t)0x7ffffffe)
    return fail(OPRAG_E_INVALID, "capacity %lld outside [1, 2^31 - 2]", (long long)desc->capacity);
  if (desc->device < 0) return fail(OPRAG_E_INVALID, "device %d < 0", desc->device);
  if (desc->reserved != 0) return fail(OPRAG_E_INVALID, "reserved field must be 0");
  if (oprag_status st = check_buf(slab_dev, "slab_dev")) return st;
  const size_t need = (size_t)desc->capacity * (size_t)desc->dim * elem_size(desc->dtype);
  if (slab_bytes < need) return fail(OPRAG_E_INVALID, "slab_bytes %zu < capacity * dim * elem = %zu", slab_bytes, need);

  int n_dev = 0;
  const hipError_t e = hipGetDeviceCount(&n_dev);
  if (e != hipSuccess) return hip_fail(e, "device count");
  if (desc->device >= n_dev) return fail(OPRAG_E_INVALID, "device %d does not exist (%d devices)", desc->device, n_dev);
  int n_cus = 0;
  const hipError_t ea = hipDeviceGetAttribute(&n_cus, hipDeviceAttributeMultiprocessorCount, desc->device);
  if (ea != hipSuccess) return hip_fail(ea, "compute unit count");
  if (n_cus < 1) return fail(OPRAG_E_DEVICE, "device %d reports %d compute units", desc->device, n_cus);
  oprag_index* idx = new oprag_index;
  idx->n_cus = n_cus;
  idx->dim = desc->dim;
  idx->dtype = desc->dtype;
  idx->device = desc->device;
  idx->capacity = desc->capacity;
  idx->slab = slab_dev;
  idx->slab_bytes = slab_bytes;
  *out = idx;
  return ok();
}

oprag_status oprag_index_destroy(oprag_index* idx) {
  if (!idx) return ok();
  if (idx->sp_mem) {
    DeviceScope ds(idx->device);
    (void)hipFree(idx->sp_mem);
  }
  delete idx;
  return ok();
}

oprag_status oprag_index_size(const oprag_index* idx, int64_t* n_rows) {
  if (oprag_status st = check_index(idx)) return st;
  if (!n_rows) return fail(OPRAG_E_INVALID, "n_rows is NULL");
  *n_rows = idx->n_rows;
  return ok();
}

oprag_status oprag_upsert(oprag_index* idx, const void* rows_dev, int32_t rows_dtype, int64_t m, void* stream,
                          int64_t* first_row) {
  if (oprag_status st = check_index(idx)) return st;
  if (m < 0) return fail(OPRAG_E_INVALID, "m = %lld < 0", (long long)m);
  if (!valid_dtype(rows_dtype)) return fail(OPRAG_E_INVALID, "rows_dtype %d is not an oprag_dtype", rows_dtype);
  if (rows_dtype != idx->dtype && !(rows_dtype == OPRAG_F32 && idx->dtype != OPRAG_F32))
    return fail(OPRAG_E_INVALID, "rows_dtype %d cannot be stored in a dtype %d index", rows_dtype, idx->dtype);
  if (m > idx->capacity - idx->n_rows)
    return fail(OPRAG_E_CAPACITY, "upsert of %lld rows exceeds capacity (%lld of %lld used)", (long long)m,
                (long long)idx->n_rows, (long long)idx->capacity);
  if (m == 0) {
    if (first_row) *first_row = idx->n_rows;
    return ok();
  }
  if (oprag_status st = check_buf(rows_dev, "rows_dev")) return st;
  DeviceScope ds(idx->device);
  if (ds.error() != hipSuccess) return hip_fail(ds.error(), "select device");
  const hipError_t e = oprag::launch_upsert(idx->slab, idx->dtype, idx->dim, idx->n_rows, rows_dev, rows_dtype, m,
                                            static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "upsert launch");
  if (first_row) *first_row = idx->n_rows;
  idx->n_rows += m;
  return ok();
}

oprag_status oprag_upsert_pooled(oprag_index* idx, const void* hidden_dev, int32_t hidden_dtype,
                                 const int32_t* lengths_dev, int64_t m, int32_t T, void* stream, int64_t* first_row) {
  if (oprag_status st = check_index(idx)) return st;
  if (m < 0) return fail(OPRAG_E_INVALID, "m = %lld < 0", (long long)m);
  if (hidden_dtype != OPRAG_BF16 && hidden_dtype != OPRAG_F32)
    return fail(OPRAG_E_INVALID, "hidden_dtype %d must be OPRAG_BF16 or OPRAG_F32", hidden_dtype);
  if (T < 1 || T > (1 << 20)) return fail(OPRAG_E_INVALID, "T = %d outside [1, 2^20]", T);
  if (m > idx->capacity - idx->n_rows)
    return fail(OPRAG_E_CAPACITY, "upsert of %lld rows exceeds capacity (%lld of %lld used)", (long long)m,
                (long long)idx->n_rows, (long long)idx->capacity);
  if (m == 0) {
    if (first_row) *first_row = idx->n_rows;
    return ok();
  }
  if (oprag_status st = check_buf(hidden_dev, "hidden_dev")) return st;
  if (oprag_status st = check_buf(lengths_dev, "lengths_dev")) return st;
  DeviceScope ds(idx->device);
  if (ds.error() != hipSuccess) return hip_fail(ds.error(), "select device");
  const hipError_t e = oprag::launch_pool_upsert(idx->slab, idx->dtype, idx->dim, idx->n_rows, hidden_dev,
                                                 hidden_dtype, lengths_dev, m, T, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "pooled upsert launch");
  if (first_row) *first_row = idx->n_rows;
  idx->n_rows += m;
  return ok();
}

oprag_status oprag_sparse_attach(oprag_index* idx, int32_t vocab, int64_t n_docs, int64_t nnz,
                                 const int64_t* term_indptr_dev, const int32_t* post_chunk_dev,
                                 const int32_t* post_tf_dev, const int32_t* doc_len_dev, float k1, float b,
                                 void* stream) {
  if (oprag_status st = check_index(idx)) return st;
  if (vocab < 1) return fail(OPRAG_E_INVALID, "vocab %d < 1", vocab);
  if (n_docs < 1 || n_docs > idx->capacity)
    return fail(OPRAG_E_INVALID, "n_docs %lld outside [1, capacity]", (long long)n_docs);
  if (nnz < 0 || nnz > (int64_t)1 << 40) return fail(OPRAG_E_INVALID, "nnz %lld out of range", (long long)nnz);
  if (!(std::isfinite(k1) && k1 >= 0.f)) return fail(OPRAG_E_INVALID, "k1 must be finite and >= 0");
  if (!(std::isfinite(b) && b >= 0.f && b <= 1.f)) return fail(OPRAG_E_INVALID, "b must be in [0, 1]");
  if (oprag_status st = check_buf(term_indptr_dev, "term_indptr_dev")) return st;
  if (oprag_status st = check_buf(doc_len_dev, "doc_len_dev")) return st;
  if (nnz > 0) {
    if (oprag_status st = check_buf(post_chunk_dev, "post_chunk_dev")) return st;
    if (oprag_status st = check_buf(post_tf_dev, "post_tf_dev")) return st;
  }
  DeviceScope ds(idx->device);
  if (ds.error() != hipSuccess) return hip_fail(ds.error(), "select device");
  hipStream_t s = static_cast<hipStream_t>(stream);
  // Validation first, with a small flag buffer of its own.
  hipError_t e = hipSuccess;
  {
    unsigned int* d_flag = nullptr;
    e = hipMalloc(&d_flag, 256);
    if (e != hipSuccess) return hip_fail(e, "sparse validation flag allocation");
    e = oprag::sparse_validate(vocab, n_docs, nnz, reinterpret_cast<const long long*>(term_indptr_dev),
                               post_chunk_dev, post_tf_dev, doc_len_dev, d_flag, s);
    unsigned int bad = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(&bad, d_flag, sizeof(bad), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    (void)hipFree(d_flag);
    if (e != hipSuccess) return hip_fail(e, "sparse index validation");
    if (bad)
      return fail(OPRAG_E_INVALID, "sparse index fails %u structural checks (indptr/chunk order/range/tf/doc_len)",
                  bad);
  }
  // Head terms: document frequency at least n_docs / 8 (and 64), the most frequent first, as
  // many as fit kMaxHead rows and kHeadBytes of dense weight rows.
  std::vector<long long> indptr((size_t)vocab + 1);
  e = hipMemcpy(indptr.data(), term_indptr_dev, indptr.size() * sizeof(long long), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "term offsets to host");
  const long long head_ld = (n_docs + 3) & ~3ll;
  std::vector<int> head;
  for (int t = 0; t < vocab; ++t) {
    const long long df = indptr[t + 1] - indptr[t];
    if (df >= 64 && 8 * df >= n_docs) head.push_back(t);
  }
  std::stable_sort(head.begin(), head.end(),
                   [&](int a, int b2) { return indptr[a + 1] - indptr[a] > indptr[b2 + 1] - indptr[b2]; });
  const long long head_cap = std::min<long long>(oprag::kMaxHead, oprag::kHeadBytes / (head_ld * 4));
  if ((long long)head.size() > head_cap) head.resize((size_t)std::max(0ll, head_cap));
  std::vector<int> hidx((size_t)vocab, -1);
  for (size_t h = 0; h < head.size(); ++h) hidx[(size_t)head[h]] = (int)h;
  const int n_head = (int)head.size();
  // Library-owned arrays: [sum u64 | idfk f32 x vocab | posting weights f32 x nnz |
  // chunk-major copy: list offsets i64 x (n_docs + 1), terms i32 x nnz, weights f32 x nnz |
  // head rows of term t i32 x vocab | head terms i32 x n_head | head rows f32 x n_head x head_ld].
  const size_t off_sum = 0, off_idf = 256;
  const size_t off_wpost = off_idf + align_up((size_t)vocab * 4);
  const size_t off_fptr = off_wpost + align_up((size_t)nnz * 4);
  const size_t off_fterm = off_fptr + align_up((size_t)(n_docs + 1) * 8);
  const size_t off_fw = off_fterm + align_up((size_t)nnz * 4);
  const size_t off_hidx = off_fw + align_up((size_t)nnz * 4);
  const size_t off_hterm = off_hidx + align_up((size_t)vocab * 4);
  const size_t off_whead = off_hterm + align_up((size_t)std::max(1, n_head) * 4);
  const size_t bytes = off_whead + align_up((size_t)n_head * (size_t)head_ld * 4);
  void* mem = nullptr;
  e = hipMalloc(&mem, bytes);
  if (e != hipSuccess) return hip_fail(e, "sparse arrays allocation");
  unsigned char* base = static_cast<unsigned char*>(mem);
  oprag::SparseIndex sp;
  sp.vocab = vocab;
  sp.n_docs = n_docs;
  sp.nnz = nnz;
  sp.term_indptr = reinterpret_cast<const long long*>(term_indptr_dev);
  sp.post_chunk = post_chunk_dev;
  sp.post_tf = post_tf_dev;
  sp.idfk = reinterpret_cast<float*>(base + off_idf);
  sp.wpost = reinterpret_cast<float*>(base + off_wpost);
  sp.fwd_ptr = reinterpret_cast<long long*>(base + off_fptr);
  sp.fwd_term = reinterpret_cast<int*>(base + off_fterm);
  sp.fwd_w = reinterpret_cast<float*>(base + off_fw);
  sp.n_head = n_head;
  sp.head_ld = head_ld;
  sp.hidx = reinterpret_cast<int*>(base + off_hidx);
  sp.whead = reinterpret_cast<float*>(base + off_whead);
  sp.k1 = k1;
  sp.b = b;
  e = hipMemcpy(sp.hidx, hidx.data(), (size_t)vocab * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess && n_head > 0)
    e = hipMemcpy(base + off_hterm, head.data(), (size_t)n_head * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = oprag::sparse_prepare(sp, doc_len_dev, reinterpret_cast<unsigned long long*>(base + off_sum), s);
  if (e == hipSuccess && n_head > 0) e = oprag::sparse_head_rows(sp, reinterpret_cast<const int*>(base + off_hterm), s);
  if (e == hipSuccess) {  // the chunk-major copy, with per-chunk counters as scratch
    int* cnt = nullptr;
    e = hipMalloc(&cnt, (size_t)n_docs * sizeof(int));
    if (e == hipSuccess) {
      e = oprag::sparse_forward(sp, cnt, s);
      const hipError_t es = hipStreamSynchronize(s);
      if (e == hipSuccess) e = es;
      (void)hipFree(cnt);
    }
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    (void)hipFree(mem);
    return hip_fail(e, "sparse index preparation");
  }
  if (sp.avgdl <= 0.0 && b > 0.f) {
    (void)hipFree(mem);
    return fail(OPRAG_E_INVALID, "all chunks are empty (avgdl = 0) while b > 0");
  }
  if (idx->sp_mem) (void)hipFree(idx->sp_mem);
  idx->sp_mem = mem;
  idx->sp = sp;
  idx->has_sparse = true;
  return ok();
}

oprag_status oprag_workspace_bytes(const oprag_index* idx, int32_t op, int64_t nq, int32_t k_dense, int32_t k_sparse,
                                   size_t* bytes) {
  if (oprag_status st = check_index(idx)) return st;
  if (!bytes) return fail(OPRAG_E_INVALID, "bytes is NULL");
  if (nq < 0) return fail(OPRAG_E_INVALID, "nq < 0");
  switch (op) {
    case OPRAG_OP_DENSE:
      if (oprag_status st = check_k(k_dense, "k_dense")) return st;
      *bytes = nq ? dense_ws(idx, nq, k_dense) : 0;
      return ok();
    case OPRAG_OP_SPARSE:
      if (oprag_status st = check_k(k_sparse, "k_sparse")) return st;
      *bytes = nq ? sparse_ws(idx, nq, k_sparse) : 0;
      return ok();
    case OPRAG_OP_HYBRID:
      if (oprag_status st = check_k(k_dense, "k_dense")) return st;
      if (oprag_status st = check_k(k_sparse, "k_sparse")) return st;
      *bytes = nq ? hybrid_ws(idx, nq, k_dense, k_sparse) : 0;
      return ok();
    case OPRAG_OP_WEIGHTED:
      *bytes = nq ? weighted_ws(idx, nq) : 0;
      return ok();
    case OPRAG_OP_DENSE_FIRST:
      if (oprag_status st = check_k(k_dense, "k_dense (n_cand)")) return st;
      *bytes = nq ? dense_first_ws(idx, nq, k_dense) : 0;
      return ok();
    default:
      return fail(OPRAG_E_INVALID, "op %d is not an oprag_op", op);
  }
}

oprag_status oprag_search_dense(const oprag_index* idx, const void* q_dev, int64_t nq, int32_t k, float* scores_dev,
                                int64_t* ids_dev, void* workspace_dev, size_t workspace_bytes, void* stream) {
  if (oprag_status st = check_index(idx)) return st;
  if (oprag_status st = check_k(k, "k")) return st;
  if (nq < 0 || nq > (int64_t)1 << 31) return fail(OPRAG_E_INVALID, "nq %lld out of range", (long long)nq);
  if (nq == 0) return ok();
  if (oprag_status st = check_buf(q_dev, "q_dev")) return st;
  if (oprag_status st = check_buf(scores_dev, "scores_dev")) return st;
  if (oprag_status st = check_buf(ids_dev, "ids_dev")) return st;
  const size_t need = dense_ws(idx, nq, k);
  if (need && (!workspace_dev || !aligned16(workspace_dev)))
    return fail(OPRAG_E_INVALID, "workspace_dev is NULL or misaligned");
  if (workspace_bytes < need) return fail(OPRAG_E_INVALID, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
  DeviceScope ds(idx->device);
  if (ds.error() != hipSuccess) return hip_fail(ds.error(), "select device");
  if (oprag_status st = do_dense(idx, q_dev, nq, k, scores_dev, ids_dev, workspace_dev, workspace_bytes,
                                 static_cast<hipStream_t>(stream)))
    return st;
  return ok();
}

oprag_status oprag_search_dense_noalloc(const oprag_index* idx, const void* q_dev, int64_t nq, int32_t k, float* scores_dev,
                                        int64_t* ids_dev, void* stream) {
  if (oprag_status st = check_index(idx)) return st;
  if (oprag_status st = check_k(k, "k")) return st;
  if (nq < 0 || nq > (int64_t)1 << 31) return fail(OPRAG_E_INVALID, "nq %lld out of range", (long long)nq);
  if (nq == 0) return ok();
  if (oprag_status st = check_buf(q_dev, "q_dev")) return st;
  if (oprag_status st = check_buf(scores_dev, "scores_dev")) return st;
  if (oprag_status st = check_buf(ids_dev, "ids_dev")) return st;
  const size_t need = dense_ws_now(idx, nq, k);
  if (need > kNoallocScratchBytes)
    return fail(OPRAG_E_CAPACITY, "search needs %zu bytes of scratch, the fixed array holds %zu (fewer queries per call)",
                need, kNoallocScratchBytes);
  DeviceScope ds(idx->device);
  if (ds.error() != hipSuccess) return hip_fail(ds.error(), "select device");
  void* ws = nullptr;
  if (oprag_status st = scratch_of(idx->device, &ws)) return st;
  if (oprag_status st = do_dense(idx, q_dev, nq, k, scores_dev, ids_dev, ws, kNoallocScratchBytes,
                                 static_cast<hipStream_t>(stream)))
    return st;
  return ok();
}

oprag_status oprag_search_sparse(const oprag_index* idx, const int32_t* qterm_indptr_dev, const int32_t* qterms_dev,
                                 int64_t nq, int32_t k, float* scores_dev, int64_t* ids_dev, void* workspace_dev,
                                 size_t workspace_bytes, void* stream) {
  if (oprag_status st = check_index(idx)) return st;
  if (!idx->has_sparse) return fail(OPRAG_E_STATE, "no sparse index attached");
  if (oprag_status st = check_k(k, "k")) return st;
  if (nq < 0 || nq > (int64_t)1 << 24) return fail(OPRAG_E_INVALID, "nq %lld out of range", (long long)nq);
  if (nq == 0) return ok();
  if (oprag_status st = check_buf(qterm_indptr_dev, "qterm_indptr_dev")) return st;
  if (!qterms_dev) return fail(OPRAG_E_INVALID, "qterms_dev is NULL");
  if (oprag_status st = check_buf(scores_dev, "scores_dev")) return st;
  if (oprag_status st = check_buf(ids_dev, "ids_dev")) return st;
  const size_t need = sparse_ws(idx, nq, k);
  if (need && (!workspace_dev || !aligned16(workspace_dev) || workspace_bytes < need))
    return fail(OPRAG_E_INVALID, "workspace missing or too small (%zu < %zu bytes)", workspace_bytes, need);
  DeviceScope ds(idx->device);
  if (ds.error() != hipSuccess) return hip_fail(ds.error(), "select device");
  const hipError_t e = oprag::launch_sparse(idx->sp, qterm_indptr_dev, qterms_dev, (int)nq, k, scores_dev,
                                            reinterpret_cast<long long*>(ids_dev), workspace_dev,
                                            static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "sparse search launch");
  return ok();
}

oprag_status oprag_rrf_fuse(const int64_t* dense_ids_dev, int32_t k_dense, const int64_t* sparse_ids_dev,
                            int32_t k_sparse, int64_t nq, int32_t rrf_k, int32_t k, float* fused_dev,
                            int64_t* ids_dev, void* stream) {
  if (oprag_status st = check_k(k_dense, "k_dense")) return st;
  if (oprag_status st = check_k(k_sparse, "k_sparse")) return st;
  if (oprag_status st = check_k(k, "k")) return st;
  if (rrf_k < 0 || rrf_k > 1000000) return fail(OPRAG_E_INVALID, "rrf_k %d outside [0, 1000000]", rrf_k);
  if (nq < 0 || nq > (int64_t)1 << 31) return fail(OPRAG_E_INVALID, "nq %lld out of range", (long long)nq);
  if (nq == 0) return ok();
  if (oprag_status st = check_buf(dense_ids_dev, "dense_ids_dev")) return st;
  if (oprag_status st = check_buf(sparse_ids_dev, "sparse_ids_dev")) return st;
  if (oprag_status st = check_buf(fused_dev, "fused_dev")) return st;
  if (oprag_status st = check_buf(ids_dev, "ids_dev")) return st;
  const hipError_t e = oprag::launch_rrf(reinterpret_cast<const long long*>(dense_ids_dev), k_dense,
                                         reinterpret_cast<const long long*>(sparse_ids_dev), k_sparse, nq, rrf_k, k,
                                         fused_dev, reinterpret_cast<long long*>(ids_dev),
                                         static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "rrf launch");
  return ok();
}

oprag_status oprag_search_hybrid(const oprag_index* idx, const void* q_dev, int64_t nq, const int32_t* qterm_indptr_dev,
                                 const int32_t* qterms_dev, int32_t k_dense, int32_t k_sparse, int32_t rrf_k, int32_t k,
                                 float* fused_dev, int64_t* ids_dev, void* workspace_dev, size_t workspace_bytes,
                                 void* stream) {
  if (oprag_status st = check_index(idx)) return st;
  if (!idx->has_sparse) return fail(OPRAG_E_STATE, "no sparse index attached");
  if (oprag_status st = check_k(k_dense, "k_dense")) return st;
  if (oprag_status st = check_k(k_sparse, "k_sparse")) return st;
  if (oprag_status st = check_k(k, "k")) return st;
  if (rrf_k < 0 || rrf_k > 1000000) return fail(OPRAG_E_INVALID, "rrf_k %d outside [0, 1000000]", rrf_k);
  if (nq < 0 || nq > (int64_t)1 << 24) return fail(OPRAG_E_INVALID, "nq %lld out of range", (long long)nq);
  if (nq == 0) return ok();
  if (oprag_status st = check_buf(q_dev, "q_dev")) return st;
  if (oprag_status st = check_buf(qterm_indptr_dev, "qterm_indptr_dev")) return st;
  if (!qterms_dev) return fail(OPRAG_E_INVALID, "qterms_dev is NULL");
  if (oprag_status st = check_buf(fused_dev, "fused_dev")) return st;
  if (oprag_status st = check_buf(ids_dev, "ids_dev")) return st;
  const size_t need = hybrid_ws(idx, nq, k_dense, k_sparse);
  if (!workspace_dev || !aligned16(workspace_dev) || workspace_bytes < need)
    return fail(OPRAG_E_INVALID, "workspace missing or too small (%zu < %zu bytes)", workspace_bytes, need);
  DeviceScope ds(idx->device);
  if (ds.error() != hipSuccess) return hip_fail(ds.error(), "select device");
  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char* w = static_cast<unsigned char*>(workspace_dev);
  int64_t* d_ids = reinterpret_cast<int64_t*>(w);
  w += align_up((size_t)nq * k_dense * 8);
  float* d_sc = reinterpret_cast<float*>(w);
  w += align_up((size_t)nq * k_dense * 4);
  int64_t* s_ids = reinterpret_cast<int64_t*>(w);
  w += align_up((size_t)nq * k_sparse * 8);
  float* s_sc = reinterpret_cast<float*>(w);
  w += align_up((size_t)nq * k_sparse * 4);
  const size_t inner = workspace_bytes - (size_t)(w - static_cast<unsigned char*>(workspace_dev));
  if (oprag_status st = do_dense(idx, q_dev, nq, k_dense, d_sc, d_ids, w, inner, s)) return st;
  if (idx->sp.n_docs <= oprag::kSparseRange) {  // one range: BM25 and the fusion in one launch
    const hipError_t e = oprag::launch_sparse_rrf(idx->sp, qterm_indptr_dev, qterms_dev, (int)nq, k_sparse,
                                                  reinterpret_cast<const long long*>(d_ids), k_dense, rrf_k, k,
                                                  fused_dev, reinterpret_cast<long long*>(ids_dev), s);
    if (e != hipSuccess) return hip_fail(e, "sparse search and fusion launch");
    return ok();
  }
  hipError_t e = oprag::launch_sparse(idx->sp, qterm_indptr_dev, qterms_dev, (int)nq, k_sparse, s_sc,
                                      reinterpret_cast<long long*>(s_ids), w, s);
  if (e != hipSuccess) return hip_fail(e, "sparse search launch");
  e = oprag::launch_rrf(reinterpret_cast<const long long*>(d_ids), k_dense, reinterpret_cast<const long long*>(s_ids),
                        k_sparse, nq, rrf_k, k, fused_dev, reinterpret_cast<long long*>(ids_dev), s);
  if (e != hipSuccess) return hip_fail(e, "rrf launch");
  return ok();
}

oprag_status oprag_search_hybrid_dense_first(const oprag_index* idx, const void* q_dev, int64_t nq,
                                             const int32_t* qterm_indptr_dev, const int32_t* qterms_dev, int32_t n_cand,
                                             int32_t rrf_k, int32_t k, float* fused_dev, int64_t* ids_dev,
                                             void* workspace_dev, size_t workspace_bytes, void* stream) {
  if (oprag_status st = check_index(idx)) return st;
  if (!idx->has_sparse) return fail(OPRAG_E_STATE, "no sparse index attached");
  if (oprag_status st = check_k(n_cand, "n_cand")) return st;
  if (oprag_status st = check_k(k, "k")) return st;
  if (rrf_k < 0 || rrf_k > 1000000) return fail(OPRAG_E_INVALID, "rrf_k %d outside [0, 1000000]", rrf_k);
  if (nq < 0 || nq > (int64_t)1 << 24) return fail(OPRAG_E_INVALID, "nq %lld out of range", (long long)nq);
  if (nq == 0) return ok();
  if (oprag_status st = check_buf(q_dev, "q_dev")) return st;
  if (oprag_status st = check_buf(qterm_indptr_dev, "qterm_indptr_dev")) return st;
  if (!qterms_dev) return fail(OPRAG_E_INVALID, "qterms_dev is NULL");
  if (oprag_status st = check_buf(fused_dev, "fused_dev")) return st;
  if (oprag_status st = check_buf(ids_dev, "ids_dev")) return st;
  const size_t need = dense_first_ws(idx, nq, n_cand);
  if (!workspace_dev || !aligned16(workspace_dev) || workspace_bytes < need)
    return fail(OPRAG_E_INVALID, "workspace missing or too small (%zu < %zu bytes)", workspace_bytes, need);
  DeviceScope ds(idx->device);
  if (ds.error() != hipSuccess) return hip_fail(ds.error(), "select device");
  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char* w = static_cast<unsigned char*>(workspace_dev);
  int64_t* c_ids = reinterpret_cast<int64_t*>(w);
  w += align_up((size_t)nq * n_cand * 8);
  float* c_sc = reinterpret_cast<float*>(w);
  w += align_up((size_t)nq * n_cand * 4);
  const size_t inner = workspace_bytes - (size_t)(w - static_cast<unsigned char*>(workspace_dev));
  if (oprag_status st = do_dense(idx, q_dev, nq, n_cand, c_sc, c_ids, w, inner, s)) return st;
  const hipError_t e =
      oprag::launch_dense_first(idx->sp, qterm_indptr_dev, qterms_dev, reinterpret_cast<const long long*>(c_ids),
                                n_cand, nq, rrf_k, k, fused_dev, reinterpret_cast<long long*>(ids_dev), s);
  if (e != hipSuccess) return hip_fail(e, "dense-first rerank launch");
  return ok();
}

oprag_status oprag_search_hybrid_weighted(const oprag_index* idx, const void* q_dev, int64_t nq,
                                          const int32_t* qterm_indptr_dev, const int32_t* qterms_dev, float w_dense,
                                          float w_lex, int32_t k, float* scores_dev, int64_t* ids_dev,
                                          void* workspace_dev, size_t workspace_bytes, void* stream) {
  if (oprag_status st = check_index(idx)) return st;
  if (!idx->has_sparse) return fail(OPRAG_E_STATE, "no sparse index attached");
  if (idx->dtype == OPRAG_F32) return fail(OPRAG_E_UNSUPPORTED, "weighted fusion needs a bf16 or fp16 index");
  if (oprag_status st = check_k(k, "k")) return st;
  if (!(std::isfinite(w_dense) && w_dense >= 0.f && std::isfinite(w_lex) && w_lex >= 0.f))
    return fail(OPRAG_E_INVALID, "weights must be finite and >= 0");
  if (nq < 0 || nq > (int64_t)1 << 24) return fail(OPRAG_E_INVALID, "nq %lld out of range", (long long)nq);
  if (nq == 0) return ok();
  if (oprag_status st = check_buf(q_dev, "q_dev")) return st;
  if (oprag_status st = check_buf(qterm_indptr_dev, "qterm_indptr_dev")) return st;
  if (!qterms_dev) return fail(OPRAG_E_INVALID, "qterms_dev is NULL");
  if (oprag_status st = check_buf(scores_dev, "scores_dev")) return st;
  if (oprag_status st = check_buf(ids_dev, "ids_dev")) return st;
  const size_t need = weighted_ws(idx, nq);
  if (!workspace_dev || !aligned16(workspace_dev) || workspace_bytes < need)
    return fail(OPRAG_E_INVALID, "workspace missing or too small (%zu < %zu bytes)", workspace_bytes, need);
  const oprag::DensePlan p = oprag::plan_dense_dump(idx->dtype, idx->dim, idx->n_rows, (int)nq, idx->n_cus);
  if (p.kernel < 0) return fail(OPRAG_E_UNSUPPORTED, "no scoring kernel for dtype %d", idx->dtype);
  DeviceScope ds(idx->device);
  if (ds.error() != hipSuccess) return hip_fail(ds.error(), "select device");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const long long ld = weighted_ld(idx);
  unsigned char* w = static_cast<unsigned char*>(workspace_dev);
  float* D = reinterpret_cast<float*>(w);
  w += align_up((size_t)nq * (size_t)ld * 4);
  float* B = reinterpret_cast<float*>(w);
  w += align_up((size_t)nq * (size_t)ld * 4);
  unsigned long long* cbuf = reinterpret_cast<unsigned long long*>(w);
  w += align_up((size_t)nq * (size_t)idx->capacity * 8);
  int* ccnt = reinterpret_cast<int*>(w);
  w += align_up((size_t)nq * 4);
  float* mm_d = reinterpret_cast<float*>(w);
  w += align_up((size_t)nq * (size_t)weighted_pd(idx, nq) * 8);
  float* mm_l = reinterpret_cast<float*>(w);
  if (p.n_chunks > weighted_pd(idx, nq)) return fail(OPRAG_E_INVALID, "internal: dump plan exceeds its bound");
  const int pl = (int)((idx->sp.n_docs + oprag::kSparseRange - 1) / oprag::kSparseRange);
  oprag::DenseArgs a;
  a.X = idx->slab;
  a.n_rows = idx->n_rows;
  a.d = idx->dim;
  a.Q = q_dev;
  a.nq = (int)nq;
  a.k = 1;
  a.dump = D;
  a.dump_ld = ld;
  a.dump_mm = mm_d;
  hipError_t e = oprag::launch_dense_dump(p, a, s);
  if (idx->n_rows <= oprag::kSparseRange && idx->sp.n_docs <= oprag::kSparseRange) {
    // one range: the BM25 kernel fuses its scores with the dense dump and selects the top k
    if (e == hipSuccess)
      e = oprag::launch_sparse_weighted(idx->sp, qterm_indptr_dev, qterms_dev, (int)nq, k, D, ld, mm_d, p.n_chunks,
                                        idx->n_rows, (double)w_dense, (double)w_lex, scores_dev,
                                        reinterpret_cast<long long*>(ids_dev), s);
    if (e != hipSuccess) return hip_fail(e, "weighted fusion launch");
    return ok();
  }
  if (e == hipSuccess)
    e = oprag::launch_sparse_dump(idx->sp, qterm_indptr_dev, qterms_dev, (int)nq, B, ld, mm_l, idx->n_rows, s);
  if (e == hipSuccess)
    e = oprag::launch_weighted_fuse(idx->n_cus, D, B, ld, idx->n_rows, std::min<long long>(idx->sp.n_docs, idx->n_rows), (int)nq,
                                    mm_d, p.n_chunks, mm_l, pl, (double)w_dense, (double)w_lex, k, cbuf, ccnt,
                                    scores_dev, reinterpret_cast<long long*>(ids_dev), s);
  if (e != hipSuccess) return hip_fail(e, "weighted fusion launch");
  return ok();
}

}  // extern "C"
