// a5 standalone and a6: the consensus error of the stored x over a column
// range, the fixed-order fp64 finalize of workgroup partials, and the
// network average.
#pragma clang fp contract(off)

#include <mutex>
#include <string>

#include "device_common.h"

// Scratch of gasloc_consensus_error_cols_noalloc: the workgroup partials, then
// the finalize's segment sums.  A file-scope device array: every GPU the
// library runs on holds its own copy for the life of the process.  In host
// code `scratch` only names the symbol; its device address on the current GPU
// comes from hipGetSymbolAddress (see noalloc_scratch below).
constexpr int kNoAllocPartials = 1 << 16;
constexpr int kNoAllocSegments = kNoAllocPartials / gasloc::kFinalizeSegment;
static __device__ __align__(256) double scratch[kNoAllocPartials + kNoAllocSegments];

namespace gasloc {
namespace {

// Columns [lo, hi) of the V-column group at idx (the others read as 0): a
// vector load when the whole group is in range.
template <int DT, int V>
__device__ __forceinline__ void load_cols(const void* base, int64_t idx, int lo, int hi, float (&o)[V]) {
  if (lo == 0 && hi == V) {
    load_params<DT, V>(base, idx, V, o);
    return;
  }
#pragma unroll
  for (int c = 0; c < V; ++c) {
    if (c >= lo && c < hi) {
      if constexpr (DT == GASLOC_BF16)
        o[c] = bf16_to_f32(static_cast<const uint16_t*>(base)[idx + c]);
      else
        o[c] = static_cast<const float*>(base)[idx + c];
    } else {
      o[c] = 0.0f;
    }
  }
}

// A thread takes a group of columns of every worker (4 fp32 or 8 bf16, i.e.
// 16 bytes; groups are aligned so every row's vector loads are, and the
// groups at the ends of the range are masked), with the loads of 8 workers
// (fp32) or 4 (bf16, twice the columns; 8 left it register-bound) in
// flight.  Per column the sums are those of the fused kernel: shifted by
// worker 0's value, fp64, workers in order.  Workgroup b takes the `per`
// consecutive steps of blockDim.x groups starting at group b * per *
// blockDim.x (tile order, as the round kernels) and writes one partial.
template <int DT>
__global__ __launch_bounds__(256) void k_consensus_error(const void* x, int64_t ld, int n,
                                                         int64_t p_begin, int64_t p_end, int per,
                                                         double* partials) {
  constexpr int V = DT == GASLOC_BF16 ? 8 : 4, R = DT == GASLOC_BF16 ? 4 : 8;
  const double inv_n = 1.0 / static_cast<double>(n);
  const int64_t base = p_begin - p_begin % V;
  const int64_t groups = (p_end - base + V - 1) / V;
  const int64_t g0 = static_cast<int64_t>(blockIdx.x) * per * blockDim.x;
  const int64_t g_end = groups - g0 < static_cast<int64_t>(per) * blockDim.x ? groups : g0 + per * blockDim.x;
  double ce = 0.0;
  for (int64_t gi = g0 + threadIdx.x; gi < g_end; gi += blockDim.x) {
    const int64_t p = base + gi * V;
    const int lo = p < p_begin ? static_cast<int>(p_begin - p) : 0;
    const int hi = p_end - p < V ? static_cast<int>(p_end - p) : V;
    double shift[V], s[V], q[V];
    {
      float v[V];
      load_cols<DT, V>(x, p, lo, hi, v);
#pragma unroll
      for (int c = 0; c < V; ++c) {
        shift[c] = static_cast<double>(v[c]);
        s[c] = 0.0;
        q[c] = 0.0;
      }
    }
    for (int i0 = 1; i0 < n; i0 += R) {
      float v[R][V];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (i0 + r >= n) break;
        load_cols<DT, V>(x, static_cast<int64_t>(i0 + r) * ld + p, lo, hi, v[r]);
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (i0 + r >= n) break;
#pragma unroll
        for (int c = 0; c < V; ++c) {
          const double d = static_cast<double>(v[r][c]) - shift[c];
          s[c] += d;
          q[c] += d * d;
        }
      }
    }
#pragma unroll
    for (int c = 0; c < V; ++c)
      if (c >= lo && c < hi) ce += q[c] - s[c] * s[c] * inv_n;
  }
  const double total = block_sum(ce);
  if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

// Fixed-order sum of `count` partials into *out (one workgroup).
__global__ __launch_bounds__(256) void k_finalize(const double* partials, int count, double* out) {
  double v = 0.0;
  for (int k = threadIdx.x; k < count; k += blockDim.x) v += partials[k];
  const double total = block_sum(v);
  if (threadIdx.x == 0) *out = total;
}

// The same for the two partial arrays of a round (consensus error, squared
// pseudo-gradients) in one launch: out[0], out[1], each in k_finalize's order.
__global__ __launch_bounds__(256) void k_finalize2(const double* a, const double* b, int count, double* out) {
  double va = 0.0, vb = 0.0;
  for (int k = threadIdx.x; k < count; k += blockDim.x) {
    va += a[k];
    vb += b[k];
  }
  double ta, tb;
  block_sum2(va, vb, ta, tb);
  if (threadIdx.x == 0) {
    out[0] = ta;
    out[1] = tb;
  }
}

// First level of the segmented finalize: workgroup s sums the partials
// [s * kFinalizeSegment, (s + 1) * kFinalizeSegment) of `a` (and of `b`
// unless it is NULL; fewer in the last segment) in k_finalize's order, into
// seg[s] (and seg[S + s]).
__global__ __launch_bounds__(256) void k_finalize_segments(const double* a, const double* b, int count,
                                                           double* seg) {
  const int begin = blockIdx.x * kFinalizeSegment;
  const int end = count - begin < kFinalizeSegment ? count : begin + kFinalizeSegment;
  double va = 0.0, vb = 0.0;
  for (int k = begin + threadIdx.x; k < end; k += blockDim.x) {
    va += a[k];
    if (b) vb += b[k];
  }
  double ta, tb;
  block_sum2(va, vb, ta, tb);
  if (threadIdx.x == 0) {
    seg[blockIdx.x] = ta;
    if (b) seg[gridDim.x + blockIdx.x] = tb;
  }
}

// a6: network average, fp64 sum in worker order, rounded to the param dtype;
// 16 bytes of columns per thread, the loads of 8 workers in flight at a time;
// workgroups in tile order, `per` steps each.
template <int DT>
__global__ __launch_bounds__(256) void k_replica_mean(const void* x, int64_t ld, int n, int64_t P, int per,
                                                      void* out) {
  constexpr int V = DT == GASLOC_BF16 ? 8 : 4, R = 8;
  const int64_t groups = (P + V - 1) / V;
  const int64_t g0 = static_cast<int64_t>(blockIdx.x) * per * blockDim.x;
  const int64_t g_end = groups - g0 < static_cast<int64_t>(per) * blockDim.x ? groups : g0 + per * blockDim.x;
  for (int64_t gi = g0 + threadIdx.x; gi < g_end; gi += blockDim.x) {
    const int64_t p = gi * V;
    const int cnt = static_cast<int>(P - p < V ? P - p : V);
    double s[V];
#pragma unroll
    for (int c = 0; c < V; ++c) s[c] = 0.0;
    for (int i0 = 0; i0 < n; i0 += R) {
      float v[R][V];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (i0 + r >= n) break;
        load_params<DT, V>(x, static_cast<int64_t>(i0 + r) * ld + p, cnt, v[r]);
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (i0 + r >= n) break;
#pragma unroll
        for (int c = 0; c < V; ++c) s[c] += static_cast<double>(v[r][c]);
      }
    }
    float mean[V], kept[V];
#pragma unroll
    for (int c = 0; c < V; ++c) mean[c] = static_cast<float>(s[c] / static_cast<double>(n));
    store_params<DT, V>(out, p, cnt, mean, kept);
  }
}

}  // namespace

int consensus_error_blocks(int dtype, int64_t p_begin, int64_t p_end, int per) {
  const int V = dtype == GASLOC_BF16 ? 8 : 4;
  const int64_t base = p_begin - p_begin % V;
  const int64_t groups = (p_end - base + V - 1) / V;
  const int64_t span = static_cast<int64_t>(per) * kReduceThreads;
  const int64_t blocks = (groups + span - 1) / span;
  return static_cast<int>(blocks < 1 ? 1 : (blocks > (int64_t(1) << 30) ? (int64_t(1) << 30) : blocks));
}

hipError_t launch_consensus_error(const void* x, int dtype, int64_t ld, int n, int64_t p_begin,
                                  int64_t p_end, int per, double* partials, hipStream_t stream) {
  const int blocks = consensus_error_blocks(dtype, p_begin, p_end, per);
  if (dtype == GASLOC_BF16)
    hipLaunchKernelGGL((k_consensus_error<GASLOC_BF16>), dim3(blocks), dim3(kReduceThreads), 0, stream, x, ld,
                       n, p_begin, p_end, per, partials);
  else
    hipLaunchKernelGGL((k_consensus_error<GASLOC_F32>), dim3(blocks), dim3(kReduceThreads), 0, stream, x, ld, n,
                       p_begin, p_end, per, partials);
  return hipGetLastError();
}

hipError_t launch_finalize_large(const double* a, int count, double* seg, double* out, hipStream_t stream) {
  if (count <= kFinalizeSegment) return launch_finalize(a, count, out, stream);
  const int segments = (count + kFinalizeSegment - 1) / kFinalizeSegment;
  hipLaunchKernelGGL(k_finalize_segments, dim3(segments), dim3(256), 0, stream, a, nullptr, count, seg);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_finalize(seg, segments, out, stream);
}

hipError_t launch_finalize(const double* partials, int count, double* out, hipStream_t stream) {
  hipLaunchKernelGGL(k_finalize, dim3(1), dim3(256), 0, stream, partials, count, out);
  return hipGetLastError();
}

hipError_t launch_finalize2(const double* a, const double* b, int count, double* out, hipStream_t stream) {
  hipLaunchKernelGGL(k_finalize2, dim3(1), dim3(256), 0, stream, a, b, count, out);
  return hipGetLastError();
}

hipError_t launch_finalize2_large(const double* a, const double* b, int count, double* seg, double* out,
                                  hipStream_t stream) {
  if (count <= kFinalizeSegment) return launch_finalize2(a, b, count, out, stream);
  const int segments = (count + kFinalizeSegment - 1) / kFinalizeSegment;
  hipLaunchKernelGGL(k_finalize_segments, dim3(segments), dim3(256), 0, stream, a, b, count, seg);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_finalize2(seg, seg + segments, segments, out, stream);
}

hipError_t launch_replica_mean(const void* x, int dtype, int64_t ld, int n, int64_t P, int per, void* out,
                               hipStream_t stream) {
  const int blocks = consensus_error_blocks(dtype, 0, P, per);
  if (dtype == GASLOC_BF16)
    hipLaunchKernelGGL((k_replica_mean<GASLOC_BF16>), dim3(blocks), dim3(kReduceThreads), 0, stream, x, ld, n, P,
                       per, out);
  else
    hipLaunchKernelGGL((k_replica_mean<GASLOC_F32>), dim3(blocks), dim3(kReduceThreads), 0, stream, x, ld, n, P,
                       per, out);
  return hipGetLastError();
}

}  // namespace gasloc

namespace {

constexpr int kNoAllocPer = 8;  // steps per workgroup, as the context's reduction on long ranges
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
double* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on the current GPU, looked up once per device
// with that device current.
hipError_t noalloc_scratch(double** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = static_cast<double*>(p);
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

gasloc_status noalloc_fail(gasloc_status st, const std::string& msg) {
  gasloc::set_thread_error("consensus_error_cols_noalloc: " + msg);
  return st;
}

}  // namespace

extern "C" gasloc_status gasloc_consensus_error_cols_noalloc(const void* x, int32_t param_dtype, int32_t n,
                                                             int64_t ld, int64_t p_begin, int64_t p_end,
                                                             double* out, void* hip_stream) {
  if (!x || (reinterpret_cast<uintptr_t>(x) & 15u)) return noalloc_fail(GASLOC_EINVAL, "x must be non-NULL and 16-byte aligned");
  if (!out || (reinterpret_cast<uintptr_t>(out) & 7u)) return noalloc_fail(GASLOC_EINVAL, "out must be non-NULL and 8-byte aligned");
  if (param_dtype != GASLOC_F32 && param_dtype != GASLOC_BF16) return noalloc_fail(GASLOC_EINVAL, "param_dtype must be F32 or BF16");
  if (n < 1 || n > gasloc::kMaxReplicas) return noalloc_fail(GASLOC_EINVAL, "n outside [1, 64]");
  const int64_t elem = param_dtype == GASLOC_BF16 ? 2 : 4;
  if (ld < 1 || (ld * elem) % 16 != 0) return noalloc_fail(GASLOC_EINVAL, "ld * sizeof(param) must be a positive multiple of 16 bytes");
  if (p_begin < 0 || p_end < p_begin || p_end > ld || p_end >= (int64_t(1) << 31))
    return noalloc_fail(GASLOC_EINVAL, "need 0 <= p_begin <= p_end <= ld and p_end < 2^31");
  const int blocks = gasloc::consensus_error_blocks(param_dtype, p_begin, p_end, kNoAllocPer);
  if (blocks > kNoAllocPartials) {
    const int64_t most = int64_t(kNoAllocPartials) * kNoAllocPer * gasloc::kReduceThreads * (elem == 2 ? 8 : 4);
    return noalloc_fail(GASLOC_EINVAL, "column range longer than the scratch allows (at most " + std::to_string(most) +
                                           " columns of this dtype per call; split the range and add the results)");
  }
  double* ptr = nullptr;
  hipError_t e = noalloc_scratch(&ptr);
  if (e != hipSuccess) return noalloc_fail(GASLOC_EDEVICE, std::string("scratch address: ") + hipGetErrorString(e));
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  e = gasloc::launch_consensus_error(x, param_dtype, ld, n, p_begin, p_end, kNoAllocPer, ptr, stream);
  if (e == hipSuccess) e = gasloc::launch_finalize_large(ptr, blocks, ptr + kNoAllocPartials, out, stream);
  if (e != hipSuccess) return noalloc_fail(GASLOC_EDEVICE, hipGetErrorString(e));
  return GASLOC_OK;
}
