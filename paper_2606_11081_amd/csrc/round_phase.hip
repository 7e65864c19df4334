// a2-a5: pseudo-gradient, outer step, neighbour mix, consensus momentum, and
// the consensus-error and squared-pseudo-gradient partials, fused.  A thread
// owns V consecutive columns of *every* worker, so each element of x, y, u,
// zp is read and written exactly once and the in-place updates cannot race.
// Phase 1 puts one value per worker in this thread's private LDS slots (no
// barrier is needed between writing and gathering them); phase 2 gathers
// the neighbours of each row through the CSR, which is staged in LDS once
// per workgroup.
//
// What a slot holds and how a row is finished depends on the round form:
//   EQ          slot z_j = x_j - eta (delta_j + mu u_j), delta_j = x_j - y_j
//               x_i = sum_k W_ik z_k [+ gamma (z_i - zp_i)]      (Eq. 1, Eq. 2)
//   ALG1        slot y_j;  delta_i = sum_k W_ik (x_i - y_k),
//               x_i = OuterOpt(x_i, delta_i)                      (Algorithm 1)
//   DADAM       slot x_j;  x_i = sum_k W_ik x_k + (y_i - x_i)     (App. C)
//   LOCAL_DADAM slot x_j;  d_i = sum_k W_ik (x_i - x_k),
//               x_i = OuterOpt(y_i, d_i)                          (App. C)
// with OuterOpt(b, d): u = mu u + d; b - eta (d + mu u) (Nesterov) or b - eta u.
#pragma clang fp contract(off)

#include "device_common.h"

namespace gasloc {
namespace {

struct CsrEntry {
  int32_t col;
  float val;
};

template <int DT, int V, int R, bool FUSED, int FORM>
__global__ __launch_bounds__(256) void k_gossip_round(GossipArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int n = a.n;
  const int nt = blockDim.x;
  const int tid = threadIdx.x;
  float* zs = reinterpret_cast<float*>(lds);  // [n][nt][V]
  const size_t z_bytes = static_cast<size_t>(n) * nt * V * sizeof(float);
  int32_t* rp = reinterpret_cast<int32_t*>(lds + z_bytes);  // [n + 1]
  const size_t rp_bytes = (static_cast<size_t>(n + 1) * sizeof(int32_t) + 7) & ~size_t(7);
  CsrEntry* ent = reinterpret_cast<CsrEntry*>(lds + z_bytes + rp_bytes);  // [nnz]

  const int nnz = a.nnz;
  for (int k = tid; k <= n; k += nt) rp[k] = a.row_ptr[k];
  for (int k = tid; k < nnz; k += nt) ent[k] = CsrEntry{a.col[k], a.val[k]};
  __syncthreads();

  constexpr bool kEq = FORM == GASLOC_FORM_EQ;
  constexpr bool kAlg1 = FORM == GASLOC_FORM_ALG1;
  constexpr bool kMixesX = FORM == GASLOC_FORM_DADAM || FORM == GASLOC_FORM_LOCAL_DADAM;
  const double inv_n = 1.0 / static_cast<double>(n);
  const int64_t groups = (a.P + V - 1) / V;
  const int64_t g_begin = static_cast<int64_t>(blockIdx.x) * a.tile_groups;
  const int64_t g_end = groups - g_begin < a.tile_groups ? groups : g_begin + a.tile_groups;
  double ce = 0.0, pg = 0.0;  // consensus error, squared pseudo-gradients
  for (int64_t gi = g_begin + tid; gi < g_end; gi += nt) {
    const int64_t p = gi * V;
    const int cnt = static_cast<int>(a.P - p < V ? a.P - p : V);
    auto slot = [&](int j) { return zs + (static_cast<size_t>(j) * nt + tid) * V; };

    // phase 1: one slot value per worker; the loads of R workers are issued
    // together before any of them is used
    for (int i0 = 0; i0 < n; i0 += R) {
      constexpr int RF = FUSED ? R : 1;
      constexpr int RU = kEq ? R : 1;
      float xv[R][V], yv[R][V], uv[RU][V];
      float gv[RF][V], mv[RF][V], vv[RF][V];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = i0 + r;
        if (i >= n) break;
        const int64_t e = static_cast<int64_t>(i) * a.ld + p;
        const bool stepped = (a.stepped >> i) & 1ull;
        if (kEq || kMixesX || !stepped) load_params<DT, V>(a.x, e, cnt, xv[r]);
        if constexpr (!kMixesX) {
          if (stepped) {
            load_params<DT, V>(a.y, e, cnt, yv[r]);
          } else {
#pragma unroll
            for (int c = 0; c < V; ++c) yv[r][c] = xv[r][c];
          }
        }
        if constexpr (FUSED) {
          if ((a.active >> i) & 1ull) {
            load_f32<V>(a.g + static_cast<int64_t>(i) * a.gld + p, cnt, gv[r]);
            load_f32<V>(a.m + e, cnt, mv[r]);
            load_f32<V>(a.v + e, cnt, vv[r]);
          }
        }
        if constexpr (kEq) {
          if (a.use_u) {
            load_f32<V>(a.u + e, cnt, uv[r]);
          } else {
#pragma unroll
            for (int c = 0; c < V; ++c) uv[r][c] = 0.0f;
          }
        }
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = i0 + r;
        if (i >= n) break;
        const int64_t e = static_cast<int64_t>(i) * a.ld + p;
        if constexpr (FUSED) {
          if ((a.active >> i) & 1ull) {
            const float s1 = a.s1[i], c2 = a.c2[i];
#pragma unroll
            for (int c = 0; c < V; ++c)
              yv[r][c] = as_stored<DT>(adamw_element(yv[r][c], gv[r][c], mv[r][c], vv[r][c], a.c_wd, a.b1,
                                                     a.omb1, a.b2, a.omb2, a.eps, s1, c2));
            store_f32<V>(a.m + e, cnt, mv[r]);
            store_f32<V>(a.v + e, cnt, vv[r]);
          }
        }
        float* out = slot(i);
        if constexpr (kEq) {
#pragma unroll
          for (int c = 0; c < V; ++c) out[c] = outer_step(xv[r][c], xv[r][c] - yv[r][c], uv[r][c], a.mu,
                                                          a.eta, a.nesterov);
          if (a.use_u) store_f32<V>(a.u + e, cnt, uv[r]);
#pragma unroll
          for (int c = 0; c < V; ++c) {
            const double d = static_cast<double>(xv[r][c] - yv[r][c]);
            if (c < cnt) pg += d * d;
          }
        } else if constexpr (kAlg1) {
#pragma unroll
          for (int c = 0; c < V; ++c) out[c] = yv[r][c];
        } else {
#pragma unroll
          for (int c = 0; c < V; ++c) out[c] = xv[r][c];
        }
      }
    }

    // phase 2: finish every row from the slots, store x (and u, zp), and
    // accumulate the consensus error of the stored x from shifted fp64 sums
    double shift[V], s[V], q[V];
    for (int i0 = 0; i0 < n; i0 += R) {
      constexpr bool kRowX = kAlg1;                                  // x_i from HBM
      constexpr bool kRowU = kAlg1 || FORM == GASLOC_FORM_LOCAL_DADAM;
      constexpr bool kRowY = kMixesX;
      float b0[R][V], b1v[(kRowU || kEq) ? R : 1][V];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = i0 + r;
        if (i >= n) break;
        const int64_t e = static_cast<int64_t>(i) * a.ld + p;
        if constexpr (kEq) {
          if (a.apply_gamma) load_f32<V>(a.zp + e, cnt, b1v[r]);
        }
        if constexpr (kRowX) load_params<DT, V>(a.x, e, cnt, b0[r]);
        if constexpr (kRowY) {
          if ((a.stepped >> i) & 1ull) {
            load_params<DT, V>(a.y, e, cnt, b0[r]);
          } else {
            const float* xi = slot(i);
#pragma unroll
            for (int c = 0; c < V; ++c) b0[r][c] = xi[c];
          }
        }
        if constexpr (kRowU) {
          if (a.use_u) {
            load_f32<V>(a.u + e, cnt, b1v[r]);
          } else {
#pragma unroll
            for (int c = 0; c < V; ++c) b1v[r][c] = 0.0f;
          }
        }
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = i0 + r;
        if (i >= n) break;
        const int64_t e = static_cast<int64_t>(i) * a.ld + p;
        const int kb = rp[i], ke = rp[i + 1];
        const float* own = slot(i);
        float res[V];
        if constexpr (kEq) {
#pragma unroll
          for (int c = 0; c < V; ++c) res[c] = 0.0f;
          for (int k = kb; k < ke; ++k) {
            const CsrEntry w = ent[k];
            const float* zj = slot(w.col);
#pragma unroll
            for (int c = 0; c < V; ++c) res[c] = res[c] + w.val * zj[c];
          }
          float zcur[V];
#pragma unroll
          for (int c = 0; c < V; ++c) zcur[c] = own[c];
          if (a.apply_gamma) {
#pragma unroll
            for (int c = 0; c < V; ++c) res[c] = res[c] + a.gamma * (zcur[c] - b1v[r][c]);
          }
          if (a.store_zp) store_f32<V>(a.zp + e, cnt, zcur);
        } else if constexpr (FORM == GASLOC_FORM_DADAM) {
#pragma unroll
          for (int c = 0; c < V; ++c) res[c] = 0.0f;
          for (int k = kb; k < ke; ++k) {
            const CsrEntry w = ent[k];
            const float* xj = slot(w.col);
#pragma unroll
            for (int c = 0; c < V; ++c) res[c] = res[c] + w.val * xj[c];
          }
#pragma unroll
          for (int c = 0; c < V; ++c) res[c] = res[c] + (b0[r][c] - own[c]);
        } else {
          // ALG1: d = sum_k W_ik (x_i - y_k), base x_i;
          // LOCAL_DADAM: d = sum_k W_ik (x_i - x_k), base y_i
          float xi[V], d[V];
#pragma unroll
          for (int c = 0; c < V; ++c) {
            xi[c] = kAlg1 ? b0[r][c] : own[c];
            d[c] = 0.0f;
          }
          for (int k = kb; k < ke; ++k) {
            const CsrEntry w = ent[k];
            const float* oj = slot(w.col);
#pragma unroll
            for (int c = 0; c < V; ++c) d[c] = d[c] + w.val * (xi[c] - oj[c]);
          }
#pragma unroll
          for (int c = 0; c < V; ++c)
            res[c] = outer_step(kAlg1 ? xi[c] : b0[r][c], d[c], b1v[r][c], a.mu, a.eta, a.nesterov);
          if (a.use_u) store_f32<V>(a.u + e, cnt, b1v[r]);
        }
        if constexpr (!kEq) {
          // pseudo-gradient x_i - y_i: ALG1 holds x_i in b0 and y_i in the
          // slot, the DAdam forms the other way round
#pragma unroll
          for (int c = 0; c < V; ++c) {
            const double d = static_cast<double>(kAlg1 ? b0[r][c] - own[c] : own[c] - b0[r][c]);
            if (c < cnt) pg += d * d;
          }
        }
        float kept[V];
        store_params<DT, V>(a.x, e, cnt, res, kept);
#pragma unroll
        for (int c = 0; c < V; ++c) {
          const double xd = static_cast<double>(kept[c]);
          if (i == 0) {
            shift[c] = xd;
            s[c] = 0.0;
            q[c] = 0.0;
          }
          const double dv = xd - shift[c];
          s[c] += dv;
          q[c] += dv * dv;
        }
      }
    }
    // sum_i (x_i - xbar)^2 = q - s^2/n with deviations taken from x_0: the
    // cancellation is bounded because q <= (n + 1) * result
#pragma unroll
    for (int c = 0; c < V; ++c)
      if (c < cnt) ce += q[c] - s[c] * s[c] * inv_n;
  }
  double total_ce, total_pg;
  block_sum2(ce, pg, total_ce, total_pg);
  if (tid == 0) {
    a.partials[blockIdx.x] = total_ce;
    a.pg_partials[blockIdx.x] = total_pg;
  }
}

// Kernel selection, shared by the launchers and the occupancy queries: F is
// called with the address of the instantiation that runs.
template <int DT, int V, int R, bool FUSED, int FORM, typename F>
hipError_t with_round_typed(F& f) {
  return f(reinterpret_cast<const void*>(&k_gossip_round<DT, V, R, FUSED, FORM>));
}

// The fused kernel carries three more streams per worker, so it batches at
// most 4 workers to stay within the register file.
template <int DT, int V, bool FUSED, int FORM, typename F>
hipError_t with_round_batched(int batch, F& f) {
  switch (batch) {
    case 1: return with_round_typed<DT, V, 1, FUSED, FORM>(f);
    case 2: return with_round_typed<DT, V, 2, FUSED, FORM>(f);
    case 8:
      if constexpr (!FUSED) return with_round_typed<DT, V, 8, FUSED, FORM>(f);
      [[fallthrough]];
    default: return with_round_typed<DT, V, 4, FUSED, FORM>(f);
  }
}

template <int DT, bool FUSED, int FORM, typename F>
hipError_t with_round_vec(const LaunchShape& s, F& f) {
  if (s.vec == 4) return with_round_batched<DT, 4, FUSED, FORM>(s.batch, f);
  if (s.vec == 2) return with_round_batched<DT, 2, FUSED, FORM>(s.batch, f);
  return with_round_batched<DT, 1, FUSED, FORM>(s.batch, f);
}

// The fused last local step exists for the forms whose slots hold the new
// local iterate or depend on it in phase 1 (EQ, ALG1).
template <int DT, typename F>
hipError_t with_round_dtype(bool fused, int form, const LaunchShape& s, F& f) {
  switch (form) {
    case GASLOC_FORM_ALG1:
      return fused ? with_round_vec<DT, true, GASLOC_FORM_ALG1>(s, f)
                   : with_round_vec<DT, false, GASLOC_FORM_ALG1>(s, f);
    case GASLOC_FORM_DADAM:
      return with_round_vec<DT, false, GASLOC_FORM_DADAM>(s, f);
    case GASLOC_FORM_LOCAL_DADAM:
      return with_round_vec<DT, false, GASLOC_FORM_LOCAL_DADAM>(s, f);
    default:
      return fused ? with_round_vec<DT, true, GASLOC_FORM_EQ>(s, f) : with_round_vec<DT, false, GASLOC_FORM_EQ>(s, f);
  }
}

template <typename F>
hipError_t with_round_kernel(int dtype, bool fused, int form, const LaunchShape& s, F& f) {
  if (dtype == GASLOC_BF16) return with_round_dtype<GASLOC_BF16>(fused, form, s, f);
  return with_round_dtype<GASLOC_F32>(fused, form, s, f);
}

}  // namespace

size_t gossip_lds_bytes(int n, int nnz, const LaunchShape& s) {
  const size_t z_bytes = static_cast<size_t>(n) * s.threads * s.vec * sizeof(float);
  const size_t rp_bytes = (static_cast<size_t>(n + 1) * sizeof(int32_t) + 7) & ~size_t(7);
  const size_t ent_bytes = static_cast<size_t>(nnz) * sizeof(CsrEntry);
  return z_bytes + rp_bytes + ent_bytes;
}

hipError_t launch_gossip_round(const GossipArgs& a, int dtype, bool fused, int form, const LaunchShape& s,
                               hipStream_t stream) {
  auto launch = [&](const void* k) { return launch_round_args(k, a, s, gossip_lds_bytes(a.n, a.nnz, s), stream); };
  return with_round_kernel(dtype, fused, form, s, launch);
}

int phase_blocks_per_cu(int dtype, bool fused, int form, const LaunchShape& s, size_t dyn_lds) {
  int blocks = 0;
  auto occupancy = [&](const void* k) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k, s.threads, dyn_lds);
  };
  return with_round_kernel(dtype, fused, form, s, occupancy) == hipSuccess ? blocks : 0;
}

}  // namespace gasloc
