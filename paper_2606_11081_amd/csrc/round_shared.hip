// a2-a5 for rounds whose rows all hold the same CSR entries (the complete
// graph, i.e. DiLoCo's average, section 3.1), EQ form (Eq. 1, Eq. 2).  The sum
//   S = sum_k W_0k z_{col_k}
// is then the same for every row, so it is accumulated once per column while
// the workers' z are produced, in ascending worker order, which is the CSR
// order of the entries (the same operands in the same order as the other
// round kernels: bit-identical).  Each row only adds its own term,
//   x_i = S + gamma (z_i - zp_i)   (the gamma term after the first round)
// kept in a statically indexed register array, so no LDS holds values: the
// kernels that keep every worker's value (or each live one) in LDS fit far
// fewer columns per CU beyond 16 workers.  A thread owns V columns of every
// worker.  (The DAdam form, whose sum is shared by equal rows too, keeps the
// planned kernel: with nothing stored before its rows, the compiler scheduled
// this kernel's loads early enough to need 352 VGPRs at 64 workers.)
#pragma clang fp contract(off)

#include <utility>

#include "device_common.h"

namespace gasloc {
namespace {

constexpr int kSharedBatch = 4;  // workers whose loads are issued together

// Workers J0 .. J0 + R - 1 (those below n): their loads issued together,
// then each one's value joins the shared sum (if its column is among the
// entries) and leaves its row term.  J0 is a template argument so that every
// index into `term` is a constant and the array stays in registers.
template <int J0, int R, int DT, int V, int NMAX, bool FUSED>
__device__ __forceinline__ void shared_workers(const GossipArgs& a, int64_t p, int cnt, float (&sum)[V],
                                               float (&term)[NMAX][V], double& pg) {
  constexpr int RF = FUSED ? R : 1;
  if (J0 >= a.n) return;
  float xv[R][V], yv[R][V], uv[R][V], zpv[R][V];
  float gv[RF][V], mv[RF][V], vv[RF][V];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = J0 + r;
    if (j >= a.n) break;
    const int64_t e = static_cast<int64_t>(j) * a.ld + p;
    const bool stepped = (a.stepped >> j) & 1ull;
    load_params<DT, V>(a.x, e, cnt, xv[r]);
    if (stepped) {
      load_params<DT, V>(a.y, e, cnt, yv[r]);
    } else {
#pragma unroll
      for (int c = 0; c < V; ++c) yv[r][c] = xv[r][c];
    }
    if constexpr (FUSED) {
      if ((a.active >> j) & 1ull) {
        load_f32<V>(a.g + static_cast<int64_t>(j) * a.gld + p, cnt, gv[r]);
        load_f32<V>(a.m + e, cnt, mv[r]);
        load_f32<V>(a.v + e, cnt, vv[r]);
      }
    }
    if (a.use_u) {
      load_f32<V>(a.u + e, cnt, uv[r]);
    } else {
#pragma unroll
      for (int c = 0; c < V; ++c) uv[r][c] = 0.0f;
    }
    if (a.apply_gamma) {
      load_f32<V>(a.zp + e, cnt, zpv[r]);
    } else {
#pragma unroll
      for (int c = 0; c < V; ++c) zpv[r][c] = 0.0f;
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = J0 + r;
    if (j >= a.n) break;
    const int64_t e = static_cast<int64_t>(j) * a.ld + p;
    if constexpr (FUSED) {
      if ((a.active >> j) & 1ull) {
        const float s1 = a.s1[j], c2 = a.c2[j];
#pragma unroll
        for (int c = 0; c < V; ++c)
          yv[r][c] = as_stored<DT>(adamw_element(yv[r][c], gv[r][c], mv[r][c], vv[r][c], a.c_wd, a.b1, a.omb1,
                                                 a.b2, a.omb2, a.eps, s1, c2));
        store_f32<V>(a.m + e, cnt, mv[r]);
        store_f32<V>(a.v + e, cnt, vv[r]);
      }
    }
    float z[V];
#pragma unroll
    for (int c = 0; c < V; ++c) {
      z[c] = outer_step(xv[r][c], xv[r][c] - yv[r][c], uv[r][c], a.mu, a.eta, a.nesterov);
      const double d = static_cast<double>(xv[r][c] - yv[r][c]);
      if (c < cnt) pg += d * d;
    }
    if (a.use_u) store_f32<V>(a.u + e, cnt, uv[r]);
    if (a.store_zp) store_f32<V>(a.zp + e, cnt, z);
    if ((a.shared_mask >> j) & 1ull) {
      const float w = a.shared_w[j];
#pragma unroll
      for (int c = 0; c < V; ++c) sum[c] = sum[c] + w * z[c];
    }
#pragma unroll
    for (int c = 0; c < V; ++c) term[J0 + r][c] = a.gamma * (z[c] - zpv[r][c]);
  }
}

// Row I (if below n): the shared sum plus its own term, stored; the shifted
// fp64 consensus-error sums of the stored value, as the other kernels.
template <int I, int DT, int V, int NMAX>
__device__ __forceinline__ void shared_row(const GossipArgs& a, int64_t p, int cnt, const float (&sum)[V],
                                           const float (&term)[NMAX][V], double (&shift)[V], double (&s)[V],
                                           double (&q)[V]) {
  if (I >= a.n) return;
  const int64_t e = static_cast<int64_t>(I) * a.ld + p;
  float res[V], kept[V];
#pragma unroll
  for (int c = 0; c < V; ++c) res[c] = a.apply_gamma ? sum[c] + term[I][c] : sum[c];
  store_params<DT, V>(a.x, e, cnt, res, kept);
#pragma unroll
  for (int c = 0; c < V; ++c) {
    const double xd = static_cast<double>(kept[c]);
    if (I == 0) {
      shift[c] = xd;
      s[c] = 0.0;
      q[c] = 0.0;
    }
    const double dv = xd - shift[c];
    s[c] += dv;
    q[c] += dv * dv;
  }
}

template <int DT, int V, int NMAX, int... I>
__device__ __forceinline__ void shared_rows(const GossipArgs& a, int64_t p, int cnt, const float (&sum)[V],
                                            const float (&term)[NMAX][V], double (&shift)[V], double (&s)[V],
                                            double (&q)[V], std::integer_sequence<int, I...>) {
  (shared_row<I, DT, V, NMAX>(a, p, cnt, sum, term, shift, s, q), ...);
}

template <int DT, int V, int NMAX, bool FUSED, int... B>
__device__ __forceinline__ void shared_column(const GossipArgs& a, int64_t p, int cnt, double& ce, double& pg,
                                              std::integer_sequence<int, B...>) {
  constexpr int R = kSharedBatch;
  float sum[V], term[NMAX][V];
#pragma unroll
  for (int c = 0; c < V; ++c) sum[c] = 0.0f;
  (shared_workers<B * R, R, DT, V, NMAX, FUSED>(a, p, cnt, sum, term, pg), ...);
  double shift[V], s[V], q[V];
  shared_rows<DT, V, NMAX>(a, p, cnt, sum, term, shift, s, q, std::make_integer_sequence<int, NMAX>{});
  const double inv_n = 1.0 / static_cast<double>(a.n);
#pragma unroll
  for (int c = 0; c < V; ++c)
    if (c < cnt) ce += q[c] - s[c] * s[c] * inv_n;
}

template <int DT, int V, int NMAX, bool FUSED>
__global__ __launch_bounds__(256) void k_gossip_shared(GossipArgs a) {
  const int nt = blockDim.x;
  const int64_t groups = (a.P + V - 1) / V;
  const int64_t g_begin = static_cast<int64_t>(blockIdx.x) * a.tile_groups;
  const int64_t g_end = groups - g_begin < a.tile_groups ? groups : g_begin + a.tile_groups;
  double ce = 0.0, pg = 0.0;  // consensus error, squared pseudo-gradients
  for (int64_t gi = g_begin + threadIdx.x; gi < g_end; gi += nt) {
    const int64_t p = gi * V;
    const int cnt = static_cast<int>(a.P - p < V ? a.P - p : V);
    shared_column<DT, V, NMAX, FUSED>(a, p, cnt, ce, pg, std::make_integer_sequence<int, NMAX / kSharedBatch>{});
  }
  double total_ce, total_pg;
  block_sum2(ce, pg, total_ce, total_pg);
  if (threadIdx.x == 0) {
    a.partials[blockIdx.x] = total_ce;
    a.pg_partials[blockIdx.x] = total_pg;
  }
}

// Kernel selection: F is called with the address of the instantiation that
// runs.  NMAX is the smallest of 16, 32, 64 that holds n, V = shared_vec(n,
// dtype): fp32 takes 2 columns per thread up to 16 workers and 1 beyond;
// bf16 takes 4, then 2 (one bf16 column per lane would make 2-byte accesses).
template <int DT, bool FUSED, typename F>
hipError_t with_shared_n(int n, F& f) {
  if constexpr (DT == GASLOC_BF16) {
    if (n <= 16) return f(reinterpret_cast<const void*>(&k_gossip_shared<DT, 4, 16, FUSED>));
    if (n <= 32) return f(reinterpret_cast<const void*>(&k_gossip_shared<DT, 2, 32, FUSED>));
    return f(reinterpret_cast<const void*>(&k_gossip_shared<DT, 2, 64, FUSED>));
  } else {
    if (n <= 16) return f(reinterpret_cast<const void*>(&k_gossip_shared<DT, 2, 16, FUSED>));
    if (n <= 32) return f(reinterpret_cast<const void*>(&k_gossip_shared<DT, 1, 32, FUSED>));
    return f(reinterpret_cast<const void*>(&k_gossip_shared<DT, 1, 64, FUSED>));
  }
}

}  // namespace

int shared_vec(int n, int dtype) {
  if (dtype == GASLOC_BF16) return n <= 16 ? 4 : 2;
  return n <= 16 ? 2 : 1;
}

hipError_t launch_gossip_shared(const GossipArgs& a, int dtype, bool fused, const LaunchShape& s, hipStream_t stream) {
  auto launch = [&](const void* k) { return launch_round_args(k, a, s, 0, stream); };
  if (dtype == GASLOC_BF16)
    return fused ? with_shared_n<GASLOC_BF16, true>(a.n, launch) : with_shared_n<GASLOC_BF16, false>(a.n, launch);
  return fused ? with_shared_n<GASLOC_F32, true>(a.n, launch) : with_shared_n<GASLOC_F32, false>(a.n, launch);
}

}  // namespace gasloc
