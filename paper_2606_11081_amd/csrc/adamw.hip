// a1: the local AdamW step of every active worker (Eq. 1 inner loop,
// App. B "Optimization": decoupled weight decay, bias-corrected moments).
#pragma clang fp contract(off)

#include "device_common.h"

namespace gasloc {
namespace {

// One workgroup per tile of 256 x 4 consecutive columns of one active worker:
// grid (tiles, n_active), tiles = ceil(P / 1024); slot blockIdx.y updates
// worker rep[slot].  The grid is not persistent: workgroups are dispatched in
// tile order, one worker row after the other, so the columns in flight at any
// moment form one compact window that sweeps each row once.  (A grid-stride
// loop over a fixed grid lets its workgroups drift apart over a row; on
// MI355X that spread the accesses over the whole row and made the launch's
// speed depend on where the buffers were placed: 25.4-30.1 ms at n = 16,
// P = 350M, against 24.3-26.0 ms for the tiles in the same processes.)
template <int DT>
__global__ __launch_bounds__(256) void k_local_adamw(AdamArgs a) {
  constexpr int V = 4;
  const int slot = blockIdx.y;
  const int64_t gi = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (gi >= (a.P + V - 1) / V) return;
  const int r = a.rep[slot];
  const bool from_x = (a.from_x >> slot) & 1ull;
  const int64_t p = gi * V;
  const int64_t e = static_cast<int64_t>(r) * a.ld + p;
  const int cnt = static_cast<int>(a.P - p < V ? a.P - p : V);
  float w[V], g[V], m[V], v[V], out[V], kept[V];
  load_params<DT, V>(from_x ? a.x : a.y, e, cnt, w);
  load_f32<V>(a.g + static_cast<int64_t>(r) * a.gld + p, cnt, g);
  load_f32<V>(a.m + e, cnt, m);
  load_f32<V>(a.v + e, cnt, v);
  const float s1 = a.s1[slot], c2 = a.c2[slot];
#pragma unroll
  for (int c = 0; c < V; ++c)
    out[c] = adamw_element(w[c], g[c], m[c], v[c], a.c_wd, a.b1, a.omb1, a.b2, a.omb2, a.eps, s1, c2);
  store_params<DT, V>(a.y, e, cnt, out, kept);
  store_f32<V>(a.m + e, cnt, m);
  store_f32<V>(a.v + e, cnt, v);
}

}  // namespace

hipError_t launch_local_adamw(const AdamArgs& a, int dtype, hipStream_t stream) {
  constexpr int64_t kTile = 256 * 4;  // columns per workgroup
  const dim3 grid(static_cast<unsigned>((a.P + kTile - 1) / kTile), a.n_active);
  if (dtype == GASLOC_BF16)
    hipLaunchKernelGGL((k_local_adamw<GASLOC_BF16>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((k_local_adamw<GASLOC_F32>), grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace gasloc
