// a1: the local AdamW step of every active worker (Eq. 1 inner loop,
// App. B "Optimization": decoupled weight decay, bias-corrected moments).
#pragma clang fp contract(off)

#include "device_common.h"

namespace gasloc {
namespace {

// grid: (blocks_per_worker, n_active); slot blockIdx.y updates worker rep[slot].
template <int DT>
__global__ __launch_bounds__(256) void k_local_adamw(AdamArgs a) {
  const int slot = blockIdx.y;
  const int r = a.rep[slot];
  const bool from_x = (a.from_x >> slot) & 1ull;
  const float s1 = a.s1[slot], c2 = a.c2[slot];
  const int64_t row = static_cast<int64_t>(r) * a.ld;
  const int64_t grow = static_cast<int64_t>(r) * a.gld;
  const void* src = from_x ? a.x : a.y;
  constexpr int V = 4;
  const int64_t groups = (a.P + V - 1) / V;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t gi = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; gi < groups;
       gi += stride) {
    const int64_t p = gi * V;
    const int cnt = static_cast<int>(a.P - p < V ? a.P - p : V);
    float w[V], g[V], m[V], v[V], out[V], kept[V];
    load_params<DT, V>(src, row + p, cnt, w);
    load_f32<V>(a.g + grow + p, cnt, g);
    load_f32<V>(a.m + row + p, cnt, m);
    load_f32<V>(a.v + row + p, cnt, v);
#pragma unroll
    for (int c = 0; c < V; ++c)
      out[c] = adamw_element(w[c], g[c], m[c], v[c], a.c_wd, a.b1, a.omb1, a.b2, a.omb2, a.eps, s1, c2);
    store_params<DT, V>(a.y, row + p, cnt, out, kept);
    store_f32<V>(a.m + row + p, cnt, m);
    store_f32<V>(a.v + row + p, cnt, v);
  }
}

}  // namespace

hipError_t launch_local_adamw(const AdamArgs& a, int dtype, int blocks_per_worker, hipStream_t stream) {
  const dim3 grid(blocks_per_worker, a.n_active);
  if (dtype == GASLOC_BF16)
    hipLaunchKernelGGL((k_local_adamw<GASLOC_BF16>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((k_local_adamw<GASLOC_F32>), grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace gasloc
