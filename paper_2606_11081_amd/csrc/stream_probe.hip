// Measurement support: a streaming kernel with the byte mix of a round
// kernel (see gasloc_probe.h), launched in tile order like the round's
// kernels, one workgroup of 64, 128 or 256 threads per tile of 4 elements
// per thread.
#pragma clang fp contract(off)

#include <string>

#include "device_common.h"
#include "gasloc_probe.h"

namespace gasloc {
namespace {

constexpr int kProbeStreams = 8;

struct ProbeArgs {
  const void* src[kProbeStreams];
  void* dst[kProbeStreams];
  int64_t count;
  uint32_t* sink;
};

template <int R32, int R16, int W32, int W16>
__global__ __launch_bounds__(256) void k_stream_probe(ProbeArgs a) {
  constexpr int V = 4;
  const int64_t p = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * V;
  if (p >= a.count) return;
  const int cnt = static_cast<int>(a.count - p < V ? a.count - p : V);
  float v[R32 + R16 > 0 ? R32 + R16 : 1][V];  // at least one row: a write-only mix reads nothing
#pragma unroll
  for (int k = 0; k < R32; ++k) load_f32<V>(static_cast<const float*>(a.src[k]) + p, cnt, v[k]);
#pragma unroll
  for (int k = 0; k < R16; ++k) load_bf16<V>(static_cast<const uint16_t*>(a.src[R32 + k]) + p, cnt, v[R32 + k]);
  float acc[V] = {};
#pragma unroll
  for (int k = 0; k < R32 + R16; ++k)
#pragma unroll
    for (int c = 0; c < V; ++c) acc[c] = acc[c] + v[k][c];
#pragma unroll
  for (int k = 0; k < W32; ++k) store_f32<V>(static_cast<float*>(a.dst[k]) + p, cnt, acc);
#pragma unroll
  for (int k = 0; k < W16; ++k) {
    float kept[V];
    store_bf16<V>(static_cast<uint16_t*>(a.dst[W32 + k]) + p, cnt, acc, kept);
  }
  if constexpr (W32 + W16 == 0) {
    if (__float_as_uint((acc[0] + acc[1]) + (acc[2] + acc[3])) == 0x7fc0deadu) *a.sink = 1u;
  }
}

template <int R32, int R16, int W32, int W16>
hipError_t launch_probe(const ProbeArgs& a, int threads, hipStream_t stream) {
  const int64_t tile = 4 * static_cast<int64_t>(threads);
  const int64_t tiles = (a.count + tile - 1) / tile;
  hipLaunchKernelGGL((k_stream_probe<R32, R16, W32, W16>), dim3(static_cast<unsigned>(tiles)), dim3(threads), 0,
                     stream, a);
  return hipGetLastError();
}

}  // namespace
}  // namespace gasloc

extern "C" gasloc_status gasloc_stream_probe(int32_t reads_f32, int32_t reads_bf16, int32_t writes_f32,
                                             int32_t writes_bf16, const void* const* src, void* const* dst,
                                             int64_t count, int32_t threads, void* sink, void* hip_stream) {
  using gasloc::ProbeArgs;
  auto bad = [](const char* msg) {
    gasloc::set_thread_error(msg);
    return GASLOC_EINVAL;
  };
  for (int32_t k : {reads_f32, reads_bf16, writes_f32, writes_bf16})
    if (k < 0 || k > 9) return bad("stream_probe: unsupported mix of streams");
  // the mix as four decimal digits: fp32 reads, bf16 reads, fp32 writes, bf16 writes
  const int code = reads_f32 * 1000 + reads_bf16 * 100 + writes_f32 * 10 + writes_bf16;
  bool ok = false;
  for (int k : {4000, 30, 1010, 4030, 3020, 3121, 2221, 7050, 6040, 5241}) ok = ok || k == code;
  if (!ok) return bad("stream_probe: unsupported mix of streams");
  if (count < 1 || count >= (int64_t(1) << 31)) return bad("stream_probe: count outside [1, 2^31)");
  if (threads != 64 && threads != 128 && threads != 256) return bad("stream_probe: threads must be 64, 128 or 256");
  if ((reads_f32 + reads_bf16 > 0 && !src) || (writes_f32 + writes_bf16 > 0 && !dst))
    return bad("stream_probe: NULL stream array");
  ProbeArgs a{};
  for (int k = 0; k < reads_f32 + reads_bf16; ++k) {
    if (!src[k] || (reinterpret_cast<uintptr_t>(src[k]) & 15u)) return bad("stream_probe: NULL or misaligned source");
    a.src[k] = src[k];
  }
  for (int k = 0; k < writes_f32 + writes_bf16; ++k) {
    if (!dst[k] || (reinterpret_cast<uintptr_t>(dst[k]) & 15u))
      return bad("stream_probe: NULL or misaligned destination");
    a.dst[k] = dst[k];
  }
  if (writes_f32 + writes_bf16 == 0 && (!sink || (reinterpret_cast<uintptr_t>(sink) & 3u)))
    return bad("stream_probe: a read-only mix needs a 4-byte-aligned sink");
  a.count = count;
  a.sink = static_cast<uint32_t*>(sink);
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  hipError_t e = hipSuccess;
  switch (code) {
    case 4000: e = gasloc::launch_probe<4, 0, 0, 0>(a, threads, s); break;
    case 30: e = gasloc::launch_probe<0, 0, 3, 0>(a, threads, s); break;
    case 1010: e = gasloc::launch_probe<1, 0, 1, 0>(a, threads, s); break;
    case 4030: e = gasloc::launch_probe<4, 0, 3, 0>(a, threads, s); break;
    case 3121: e = gasloc::launch_probe<3, 1, 2, 1>(a, threads, s); break;
    case 2221: e = gasloc::launch_probe<2, 2, 2, 1>(a, threads, s); break;
    case 3020: e = gasloc::launch_probe<3, 0, 2, 0>(a, threads, s); break;
    case 7050: e = gasloc::launch_probe<7, 0, 5, 0>(a, threads, s); break;
    case 6040: e = gasloc::launch_probe<6, 0, 4, 0>(a, threads, s); break;
    default: e = gasloc::launch_probe<5, 2, 4, 1>(a, threads, s); break;
  }
  if (e != hipSuccess) {
    gasloc::set_thread_error(std::string("stream_probe: ") + hipGetErrorString(e));
    return GASLOC_EDEVICE;
  }
  return GASLOC_OK;
}
