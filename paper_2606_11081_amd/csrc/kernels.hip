// HIP kernels of the GASLoC round for CDNA4 (gfx950).
//
// Every kernel here streams [n, P] buffers once: the path is HBM-bandwidth
// bound (well under 2 flop per byte), so the kernels use the vector ALU only
// (no MFMA), 16-byte-per-lane loads and stores where the dtype allows, and a
// grid-stride loop over column groups.
//
// Floating-point contract: no contraction (each product and sum is rounded
// on its own), correctly rounded fp32 division and square root (HIP's
// default), fp64 for every reduction.
#pragma clang fp contract(off)

#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace gasloc {
namespace {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// parameter storage
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// binary32 -> bfloat16, round to nearest, ties to even; NaN stays a quiet NaN
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// 16/8/4-byte register vectors for global memory traffic
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Streaming data is touched once per kernel, so the vector accesses carry the
// non-temporal hint (measured 2-4% faster on the n=16, P=350M round than
// plain accesses).  Build with -DGASLOC_NONTEMPORAL=0 to drop the hint.
#ifndef GASLOC_NONTEMPORAL
#define GASLOC_NONTEMPORAL 1
#endif
template <typename T>
__device__ __forceinline__ T ld_stream(const T* p) {
#if GASLOC_NONTEMPORAL
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}
template <typename T>
__device__ __forceinline__ void st_stream(T* p, T v) {
#if GASLOC_NONTEMPORAL
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

// Load V consecutive fp32 values; `cnt` < V only for the ragged last group of
// a row, which is read element by element.
template <int V>
__device__ __forceinline__ void load_f32(const float* p, int cnt, float (&o)[V]) {
  if (cnt == V) {
    if constexpr (V == 4) {
      const f32x4 t = ld_stream(reinterpret_cast<const f32x4*>(p));
      o[0] = t.x; o[1] = t.y; o[2] = t.z; o[3] = t.w;
    } else if constexpr (V == 2) {
      const f32x2 t = ld_stream(reinterpret_cast<const f32x2*>(p));
      o[0] = t.x; o[1] = t.y;
    } else {
      o[0] = ld_stream(p);
    }
  } else {
#pragma unroll
    for (int c = 0; c < V; ++c) o[c] = c < cnt ? p[c] : 0.0f;
  }
}

template <int V>
__device__ __forceinline__ void store_f32(float* p, int cnt, const float (&o)[V]) {
  if (cnt == V) {
    if constexpr (V == 4) {
      st_stream(reinterpret_cast<f32x4*>(p), f32x4{o[0], o[1], o[2], o[3]});
    } else if constexpr (V == 2) {
      st_stream(reinterpret_cast<f32x2*>(p), f32x2{o[0], o[1]});
    } else {
      st_stream(p, o[0]);
    }
  } else {
#pragma unroll
    for (int c = 0; c < V; ++c)
      if (c < cnt) p[c] = o[c];
  }
}

template <int V>
__device__ __forceinline__ void load_bf16(const uint16_t* p, int cnt, float (&o)[V]) {
  if (cnt == V) {
    if constexpr (V == 8) {
      const u32x4 t = ld_stream(reinterpret_cast<const u32x4*>(p));
      o[0] = bf16_to_f32(t.x & 0xffffu); o[1] = bf16_to_f32(t.x >> 16);
      o[2] = bf16_to_f32(t.y & 0xffffu); o[3] = bf16_to_f32(t.y >> 16);
      o[4] = bf16_to_f32(t.z & 0xffffu); o[5] = bf16_to_f32(t.z >> 16);
      o[6] = bf16_to_f32(t.w & 0xffffu); o[7] = bf16_to_f32(t.w >> 16);
    } else if constexpr (V == 4) {
      const u32x2 t = ld_stream(reinterpret_cast<const u32x2*>(p));
      o[0] = bf16_to_f32(t.x & 0xffffu); o[1] = bf16_to_f32(t.x >> 16);
      o[2] = bf16_to_f32(t.y & 0xffffu); o[3] = bf16_to_f32(t.y >> 16);
    } else if constexpr (V == 2) {
      const uint32_t t = ld_stream(reinterpret_cast<const uint32_t*>(p));
      o[0] = bf16_to_f32(t & 0xffffu); o[1] = bf16_to_f32(t >> 16);
    } else {
      o[0] = bf16_to_f32(*p);
    }
  } else {
#pragma unroll
    for (int c = 0; c < V; ++c) o[c] = c < cnt ? bf16_to_f32(p[c]) : 0.0f;
  }
}

// Rounds to bf16, stores, and returns the stored values as fp32 in `kept`.
template <int V>
__device__ __forceinline__ void store_bf16(uint16_t* p, int cnt, const float (&o)[V], float (&kept)[V]) {
  uint32_t h[V];
#pragma unroll
  for (int c = 0; c < V; ++c) {
    h[c] = f32_to_bf16(o[c]);
    kept[c] = bf16_to_f32(h[c]);
  }
  if (cnt == V) {
    if constexpr (V == 8) {
      st_stream(reinterpret_cast<u32x4*>(p), u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                                                   h[6] | (h[7] << 16)});
    } else if constexpr (V == 4) {
      st_stream(reinterpret_cast<u32x2*>(p), u32x2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)});
    } else if constexpr (V == 2) {
      st_stream(reinterpret_cast<uint32_t*>(p), h[0] | (h[1] << 16));
    } else {
      *p = static_cast<uint16_t>(h[0]);
    }
  } else {
#pragma unroll
    for (int c = 0; c < V; ++c)
      if (c < cnt) p[c] = static_cast<uint16_t>(h[c]);
  }
}

template <int DT, int V>
__device__ __forceinline__ void load_params(const void* base, int64_t idx, int cnt, float (&o)[V]) {
  if constexpr (DT == GASLOC_BF16)
    load_bf16<V>(static_cast<const uint16_t*>(base) + idx, cnt, o);
  else
    load_f32<V>(static_cast<const float*>(base) + idx, cnt, o);
}

template <int DT, int V>
__device__ __forceinline__ void store_params(void* base, int64_t idx, int cnt, const float (&o)[V],
                                             float (&kept)[V]) {
  if constexpr (DT == GASLOC_BF16) {
    store_bf16<V>(static_cast<uint16_t*>(base) + idx, cnt, o, kept);
  } else {
    store_f32<V>(static_cast<float*>(base) + idx, cnt, o);
#pragma unroll
    for (int c = 0; c < V; ++c) kept[c] = o[c];
  }
}

// The value a store to the parameter dtype keeps (RNE to bf16, or fp32 as is).
template <int DT>
__device__ __forceinline__ float as_stored(float v) {
  if constexpr (DT == GASLOC_BF16)
    return bf16_to_f32(f32_to_bf16(v));
  else
    return v;
}

// ---------------------------------------------------------------------------
// reductions: fixed-order DPP scan inside the wave, then the waves of the
// workgroup
// ---------------------------------------------------------------------------

// v from the lane `k` places lower in the same 16-lane row (DPP row_shr:k),
// 0 for the first k lanes of each row.  A double moves as two 32-bit halves.
template <int K>
__device__ __forceinline__ double row_shr(double v) {
  const uint64_t bits = static_cast<uint64_t>(__double_as_longlong(v));
  const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(bits)), 0x110 + K, 0xf, 0xf,
                                             true);
  const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(bits >> 32)), 0x110 + K, 0xf,
                                             0xf, true);
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) |
                                                     static_cast<uint32_t>(lo)));
}

__device__ __forceinline__ double read_lane(double v, int lane) {
  const uint64_t bits = static_cast<uint64_t>(__double_as_longlong(v));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(bits)), lane));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(bits >> 32)), lane));
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}

// Sum over the wave (all 64 lanes active), the same in every lane: an
// inclusive scan inside each 16-lane row with DPP row shifts (lane 15 of a
// row then holds the row's sum), and the four row sums added in row order.
// The order of additions is fixed, so the result is deterministic.
__device__ __forceinline__ double wave_sum(double v) {
  v += row_shr<1>(v);
  v += row_shr<2>(v);
  v += row_shr<4>(v);
  v += row_shr<8>(v);
  return ((read_lane(v, 15) + read_lane(v, 31)) + read_lane(v, 47)) + read_lane(v, 63);
}

// Sum of `v` over the workgroup, valid in thread 0.
__device__ __forceinline__ double block_sum(double v) {
  __shared__ double wave_part[1024 / kWave];
  v = wave_sum(v);
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  if (lane == 0) wave_part[wave] = v;
  __syncthreads();
  double total = 0.0;
  if (threadIdx.x == 0) {
    const int waves = (blockDim.x + kWave - 1) / kWave;
    for (int w = 0; w < waves; ++w) total += wave_part[w];
  }
  return total;
}

// Sums of `a` and `b` over the workgroup, valid in thread 0 (the round
// kernels' consensus-error and pseudo-gradient partials).
__device__ __forceinline__ void block_sum2(double a, double b, double& ta, double& tb) {
  __shared__ double wave_part2[2][1024 / kWave];
  a = wave_sum(a);
  b = wave_sum(b);
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  if (lane == 0) {
    wave_part2[0][wave] = a;
    wave_part2[1][wave] = b;
  }
  __syncthreads();
  ta = 0.0;
  tb = 0.0;
  if (threadIdx.x == 0) {
    const int waves = (blockDim.x + kWave - 1) / kWave;
    for (int w = 0; w < waves; ++w) {
      ta += wave_part2[0][w];
      tb += wave_part2[1][w];
    }
  }
}

// ---------------------------------------------------------------------------
// a1: local AdamW step
// ---------------------------------------------------------------------------

__device__ __forceinline__ float adamw_element(float y, float g, float& m, float& v, float c_wd,
                                               float b1, float omb1, float b2, float omb2,
                                               float eps, float s1, float c2) {
  const float w = y * c_wd;
  m = b1 * m + omb1 * g;
  v = b2 * v + omb2 * (g * g);
  const float d = sqrtf(v) / c2 + eps;
  return w - s1 * (m / d);
}

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

// ---------------------------------------------------------------------------
// a2-a5: pseudo-gradient, outer step, neighbour mix, consensus momentum, and
// the consensus-error and squared-pseudo-gradient partials, fused.  A thread
// owns V consecutive columns of *every* worker, so each element of x, y, u,
// zp is read and written exactly once and the in-place updates cannot race.  Phase 1 puts one value
// per worker in this thread's private LDS slots (no barrier is needed
// between writing and gathering them); phase 2 gathers the neighbours of
// each row through the CSR, which is staged in LDS once per workgroup.
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
// ---------------------------------------------------------------------------

struct CsrEntry {
  int32_t col;
  float val;
};

__device__ __forceinline__ float outer_step(float base, float d, float& u, float mu, float eta,
                                            int nesterov) {
  u = mu * u + d;
  const float step = nesterov ? d + mu * u : u;
  return base - eta * step;
}

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
  const int64_t stride = static_cast<int64_t>(gridDim.x) * nt;
  double ce = 0.0, pg = 0.0;  // consensus error, squared pseudo-gradients
  for (int64_t gi = static_cast<int64_t>(blockIdx.x) * nt + tid; gi < groups; gi += stride) {
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

// ---------------------------------------------------------------------------
// A round of any form with a host-planned visit order (plan.cpp).  Each
// super-step computes the slot values (z for EQ, the live local iterate for
// ALG1, x for the DAdam forms) of the workers its rows read first (at most R
// of them) into free LDS slots, then emits up to kPlanRows rows.  LDS holds
// `slots` values per column instead of n, so sparse graphs keep many more
// columns in flight per CU.  Per element the arithmetic is exactly that of
// k_gossip_round<..., FORM>.
//
// The plan is the same for every column, so it is read through the scalar
// cache (constant address space): worker and slot indices, counts and weights
// are wave-uniform and all control flow is scalar.  The loads of the next
// super-step (of this column group, or the first of the next group) are issued
// before the current one is computed, so a wave keeps one super-step of
// operands in flight while it works; they are held as raw words and decoded at
// their use, which keeps the loads outstanding until then.
//
// Plan words: [S, start_0 .. start_{S-1}], super-step at start_s:
//   npre, nrows, (worker, slot) x npre, row x nrows,
//   then per row: nent, own_slot, (slot, weight bits) x nent, or
//   kPlanReuseMix, own_slot (EQ, DAdam: the previous summed row's sum).
// ---------------------------------------------------------------------------

typedef const __attribute__((address_space(4))) int32_t plan_word;

// 32-bit words holding V values of dtype DT as stored
template <int DT, int V>
struct RawWords {
  static constexpr int count = DT == GASLOC_BF16 ? (V + 1) / 2 : V;
};

template <int DT, int V>
__device__ __forceinline__ void load_raw(const void* base, int64_t idx, int cnt,
                                         uint32_t (&w)[RawWords<DT, V>::count]) {
  if constexpr (DT == GASLOC_BF16) {
    const uint16_t* p = static_cast<const uint16_t*>(base) + idx;
    if (cnt == V) {
      if constexpr (V == 4) {
        const u32x2 t = ld_stream(reinterpret_cast<const u32x2*>(p));
        w[0] = t.x;
        w[1] = t.y;
      } else if constexpr (V == 2) {
        w[0] = ld_stream(reinterpret_cast<const uint32_t*>(p));
      } else {
        w[0] = *p;
      }
    } else {
#pragma unroll
      for (int k = 0; k < RawWords<DT, V>::count; ++k) w[k] = 0u;
#pragma unroll
      for (int c = 0; c < V; ++c)
        if (c < cnt) w[c / 2] |= static_cast<uint32_t>(p[c]) << (16 * (c & 1));
    }
  } else {
    const float* p = static_cast<const float*>(base) + idx;
    if (cnt == V) {
      if constexpr (V == 4) {
        const f32x4 t = ld_stream(reinterpret_cast<const f32x4*>(p));
        w[0] = __float_as_uint(t.x);
        w[1] = __float_as_uint(t.y);
        w[2] = __float_as_uint(t.z);
        w[3] = __float_as_uint(t.w);
      } else if constexpr (V == 2) {
        const f32x2 t = ld_stream(reinterpret_cast<const f32x2*>(p));
        w[0] = __float_as_uint(t.x);
        w[1] = __float_as_uint(t.y);
      } else {
        w[0] = __float_as_uint(ld_stream(p));
      }
    } else {
#pragma unroll
      for (int c = 0; c < V; ++c) w[c] = 0u;
#pragma unroll
      for (int c = 0; c < V; ++c)
        if (c < cnt) w[c] = __float_as_uint(p[c]);
    }
  }
}

template <int DT, int V>
__device__ __forceinline__ void decode_raw(const uint32_t (&w)[RawWords<DT, V>::count], float (&o)[V]) {
#pragma unroll
  for (int c = 0; c < V; ++c) {
    if constexpr (DT == GASLOC_BF16)
      o[c] = bf16_to_f32((w[c / 2] >> (16 * (c & 1))) & 0xffffu);
    else
      o[c] = __uint_as_float(w[c]);
  }
}

// Operands of one super-step, loaded ahead of their use:
//   pa, pb, pu: the new slot workers' x, y, u (EQ); y or x (ALG1); x (the
//               DAdam forms).  pb and pu are used by EQ only.
//   ra, rf:     the rows' x (ALG1) or y (DAdam forms), and zp (EQ) or u
//               (ALG1, Local-DAdam).
// The fused AdamW operands (g, m, v) are not staged: two super-steps of them
// would not fit the register budget of the occupancy the LDS allows, so they
// are loaded when the super-step is computed (with the next super-step's
// loads already in flight).
template <int DT, int V, int R>
struct Staged {
  static constexpr int PW = RawWords<DT, V>::count;
  uint32_t pa[R][PW], pb[R][PW];
  uint32_t pu[R][V];
  uint32_t ra[kPlanRows][PW];
  uint32_t rf[kPlanRows][V];
};

// TAIL: the workgroup's columns may run past P (per-thread cnt < V); else
// every thread has V columns and the accesses need no per-lane branches.
template <int DT, int V, int R, int FORM, bool TAIL>
__device__ __forceinline__ void planned_issue(const GossipArgs& a, plan_word* ops, int st, int64_t p, int cnt_tail,
                                              Staged<DT, V, R>& b) {
  constexpr bool kEq = FORM == GASLOC_FORM_EQ;
  constexpr bool kAlg1 = FORM == GASLOC_FORM_ALG1;
  const int cnt = TAIL ? cnt_tail : V;
  const int at = ops[1 + st];
  const int npre = ops[at], nrows = ops[at + 1];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r >= npre) break;
    const int j = ops[at + 2 + 2 * r];
    const int64_t e = static_cast<int64_t>(j) * a.ld + p;
    const bool stepped = (a.stepped >> j) & 1ull;
    if constexpr (kEq) {
      load_raw<DT, V>(a.x, e, cnt, b.pa[r]);
      if (stepped) load_raw<DT, V>(a.y, e, cnt, b.pb[r]);
      if (a.use_u) load_raw<GASLOC_F32, V>(a.u, e, cnt, b.pu[r]);
    } else if constexpr (kAlg1) {
      load_raw<DT, V>(stepped ? a.y : a.x, e, cnt, b.pa[r]);
    } else {
      load_raw<DT, V>(a.x, e, cnt, b.pa[r]);
    }
  }
  const int rows_at = at + 2 + 2 * npre;
#pragma unroll
  for (int rr = 0; rr < kPlanRows; ++rr) {
    if (rr >= nrows) break;
    const int row = ops[rows_at + rr];
    const int64_t er = static_cast<int64_t>(row) * a.ld + p;
    if constexpr (kEq) {
      if (a.apply_gamma) load_raw<GASLOC_F32, V>(a.zp, er, cnt, b.rf[rr]);
    } else if constexpr (kAlg1) {
      load_raw<DT, V>(a.x, er, cnt, b.ra[rr]);
      if (a.use_u) load_raw<GASLOC_F32, V>(a.u, er, cnt, b.rf[rr]);
    } else {
      if ((a.stepped >> row) & 1ull) load_raw<DT, V>(a.y, er, cnt, b.ra[rr]);
      if (FORM == GASLOC_FORM_LOCAL_DADAM && a.use_u) load_raw<GASLOC_F32, V>(a.u, er, cnt, b.rf[rr]);
    }
  }
}

// Running consensus-error sums of one column group (shifted by its first
// stored row, as in k_gossip_round); `fresh` until that row is stored.  pg:
// this thread's running sum of squared pseudo-gradients x_i - y_i.  mix: the
// neighbour sum of the last row that summed its entries, taken by the rows
// the plan marks kPlanReuseMix.
template <int V>
struct CeSums {
  double shift[V], s[V], q[V];
  bool fresh;
  double pg;
  float mix[V];
};

template <int DT, int V, int R, bool FUSED, int FORM, bool TAIL>
__device__ __forceinline__ void planned_consume(const GossipArgs& a, plan_word* ops, int st, int64_t p,
                                                int cnt_tail, const Staged<DT, V, R>& b, float* mine,
                                                int slot_stride, CeSums<V>& cs) {
  constexpr bool kEq = FORM == GASLOC_FORM_EQ;
  constexpr bool kAlg1 = FORM == GASLOC_FORM_ALG1;
  const int cnt = TAIL ? cnt_tail : V;
  const int at = ops[1 + st];
  const int npre = ops[at], nrows = ops[at + 1];
  if (st == 0) cs.fresh = true;
  constexpr int RF = FUSED ? R : 1;
  uint32_t gw[RF][V], mw[RF][V], vw[RF][V];
  if constexpr (FUSED) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (r >= npre) break;
      const int j = ops[at + 2 + 2 * r];
      if ((a.active >> j) & 1ull) {
        const int64_t e = static_cast<int64_t>(j) * a.ld + p;
        load_raw<GASLOC_F32, V>(a.g, static_cast<int64_t>(j) * a.gld + p, cnt, gw[r]);
        load_raw<GASLOC_F32, V>(a.m, e, cnt, mw[r]);
        load_raw<GASLOC_F32, V>(a.v, e, cnt, vw[r]);
      }
    }
  }
  // slot values of the workers first read in this super-step: z (EQ), the
  // live (fused: new) local iterate (ALG1), x (DAdam forms)
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r >= npre) break;
    const int j = ops[at + 2 + 2 * r];
    const int slot = ops[at + 3 + 2 * r];
    const int64_t e = static_cast<int64_t>(j) * a.ld + p;
    const bool stepped = (a.stepped >> j) & 1ull;
    float* out = mine + slot * slot_stride;
    float xv[V], yv[V];
    if constexpr (kEq) {
      decode_raw<DT, V>(b.pa[r], xv);
      if (stepped) {
        decode_raw<DT, V>(b.pb[r], yv);
      } else {
#pragma unroll
        for (int c = 0; c < V; ++c) yv[c] = xv[c];
      }
    } else {
      decode_raw<DT, V>(b.pa[r], yv);  // ALG1: y (x if not stepped); DAdam forms: x
    }
    if constexpr (FUSED) {
      if ((a.active >> j) & 1ull) {
        float gv[V], mv[V], vv[V];
        decode_raw<GASLOC_F32, V>(gw[r], gv);
        decode_raw<GASLOC_F32, V>(mw[r], mv);
        decode_raw<GASLOC_F32, V>(vw[r], vv);
        const float s1 = a.s1[j], c2 = a.c2[j];
#pragma unroll
        for (int c = 0; c < V; ++c)
          yv[c] = as_stored<DT>(adamw_element(yv[c], gv[c], mv[c], vv[c], a.c_wd, a.b1, a.omb1, a.b2, a.omb2,
                                              a.eps, s1, c2));
        store_f32<V>(a.m + e, cnt, mv);
        store_f32<V>(a.v + e, cnt, vv);
      }
    }
    if constexpr (kEq) {
      float uv[V];
      if (a.use_u) {
        decode_raw<GASLOC_F32, V>(b.pu[r], uv);
      } else {
#pragma unroll
        for (int c = 0; c < V; ++c) uv[c] = 0.0f;
      }
#pragma unroll
      for (int c = 0; c < V; ++c) out[c] = outer_step(xv[c], xv[c] - yv[c], uv[c], a.mu, a.eta, a.nesterov);
      if (a.use_u) store_f32<V>(a.u + e, cnt, uv);
#pragma unroll
      for (int c = 0; c < V; ++c) {
        const double d = static_cast<double>(xv[c] - yv[c]);
        if (c < cnt) cs.pg += d * d;
      }
    } else {
#pragma unroll
      for (int c = 0; c < V; ++c) out[c] = yv[c];
    }
  }

  // the rows, each summing its CSR entries in order (four entries' LDS reads
  // in flight at a time):
  //   EQ:          x_r = sum_k W_rk z_k (+ gamma (z_r - zp_r)), zp_r = z_r
  //   ALG1:        d = sum_k W_rk (x_r - y_k), outer step from x_r
  //   DAdam:       x_r = sum_k W_rk x_k + (y_r - x_r)
  //   Local-DAdam: d = sum_k W_rk (x_r - x_k), outer step from y_r
  // In EQ and DAdam the sum does not depend on the row, so a row with the
  // entries of the row summed before it takes that sum (kPlanReuseMix).
  const int rows_at = at + 2 + 2 * npre;
  int pos = rows_at + nrows;
#pragma unroll
  for (int rr = 0; rr < kPlanRows; ++rr) {
    if (rr >= nrows) break;
    const int row = ops[rows_at + rr];
    const int nent = ops[pos];
    const int64_t er = static_cast<int64_t>(row) * a.ld + p;
    float own[V];
    {
      const float* zo = mine + ops[pos + 1] * slot_stride;
#pragma unroll
      for (int c = 0; c < V; ++c) own[c] = zo[c];
    }
    // xi: the value the differences are taken from (ALG1, Local-DAdam)
    float xi[V];
    if constexpr (kAlg1) {
      decode_raw<DT, V>(b.ra[rr], xi);
    } else {
#pragma unroll
      for (int c = 0; c < V; ++c) xi[c] = own[c];
    }
    constexpr bool kDiff = kAlg1 || FORM == GASLOC_FORM_LOCAL_DADAM;
    // a reusing row starts from the kept sum and adds no entries
    const bool reuse = !kDiff && nent == kPlanReuseMix;
    const int count = reuse ? 0 : nent;
    float acc[V];
#pragma unroll
    for (int c = 0; c < V; ++c) acc[c] = reuse ? cs.mix[c] : 0.0f;
    for (int k0 = 0; k0 < count; k0 += 4) {
      float zk[4][V], wk[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (k0 + t >= count) break;
        const float* src = mine + ops[pos + 2 + 2 * (k0 + t)] * slot_stride;
        wk[t] = __int_as_float(ops[pos + 3 + 2 * (k0 + t)]);
#pragma unroll
        for (int c = 0; c < V; ++c) zk[t][c] = src[c];
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (k0 + t >= count) break;
#pragma unroll
        for (int c = 0; c < V; ++c) acc[c] = acc[c] + wk[t] * (kDiff ? xi[c] - zk[t][c] : zk[t][c]);
      }
    }
    pos += 2 + 2 * count;
    if constexpr (!kDiff) {
#pragma unroll
      for (int c = 0; c < V; ++c) cs.mix[c] = acc[c];
    }
    float res[V];
    if constexpr (kEq) {
      if (a.apply_gamma) {
        float zpv[V];
        decode_raw<GASLOC_F32, V>(b.rf[rr], zpv);
#pragma unroll
        for (int c = 0; c < V; ++c) acc[c] = acc[c] + a.gamma * (own[c] - zpv[c]);
      }
      if (a.store_zp) store_f32<V>(a.zp + er, cnt, own);
#pragma unroll
      for (int c = 0; c < V; ++c) res[c] = acc[c];
    } else {
      // ALG1: x_r; DAdam forms: y_r, or x_r itself for a worker without local
      // steps
      float base[V];
      if constexpr (kAlg1) {
#pragma unroll
        for (int c = 0; c < V; ++c) base[c] = xi[c];
      } else if ((a.stepped >> row) & 1ull) {
        decode_raw<DT, V>(b.ra[rr], base);
      } else {
#pragma unroll
        for (int c = 0; c < V; ++c) base[c] = own[c];
      }
      // pseudo-gradient x_r - y_r: ALG1 holds y_r in the slot, the DAdam
      // forms hold x_r there
#pragma unroll
      for (int c = 0; c < V; ++c) {
        const double d = static_cast<double>(kAlg1 ? base[c] - own[c] : own[c] - base[c]);
        if (c < cnt) cs.pg += d * d;
      }
      if constexpr (FORM == GASLOC_FORM_DADAM) {
#pragma unroll
        for (int c = 0; c < V; ++c) res[c] = acc[c] + (base[c] - own[c]);
      } else {
        float uv[V];
        if (a.use_u) {
          decode_raw<GASLOC_F32, V>(b.rf[rr], uv);
        } else {
#pragma unroll
          for (int c = 0; c < V; ++c) uv[c] = 0.0f;
        }
#pragma unroll
        for (int c = 0; c < V; ++c) res[c] = outer_step(base[c], acc[c], uv[c], a.mu, a.eta, a.nesterov);
        if (a.use_u) store_f32<V>(a.u + er, cnt, uv);
      }
    }
    float kept[V];
    store_params<DT, V>(a.x, er, cnt, res, kept);
#pragma unroll
    for (int c = 0; c < V; ++c) {
      const double xd = static_cast<double>(kept[c]);
      if (cs.fresh) {
        cs.shift[c] = xd;
        cs.s[c] = 0.0;
        cs.q[c] = 0.0;
      }
      const double dv = xd - cs.shift[c];
      cs.s[c] += dv;
      cs.q[c] += dv * dv;
    }
    cs.fresh = false;
  }
}

template <int DT, int V, int R, bool FUSED, int FORM>
__global__ __launch_bounds__(256) void k_gossip_planned(GossipArgs a) {
  extern __shared__ __align__(16) float zs[];  // [slots][nt][V]
  plan_word* ops = (plan_word*)(a.ops);  // address-space cast: read-only for the whole launch
  const int nt = blockDim.x;
  const int tid = threadIdx.x;
  const int steps = ops[0];
  const double inv_n = 1.0 / static_cast<double>(a.n);
  const int slot_stride = nt * V;
  float* mine = zs + tid * V;

  // column groups blockIdx.x * nt + it * (gridDim.x * nt) + tid, it < iters:
  // the same count for every thread of the workgroup, so control stays
  // uniform.  Every iteration but possibly the last gives each thread V
  // columns; in that last one threads past P see cnt < V (0 beyond the end)
  const int64_t groups = (a.P + V - 1) / V;
  const int64_t whole = a.P / V;  // groups with V columns
  const int64_t span = static_cast<int64_t>(gridDim.x) * nt;
  const int64_t first = static_cast<int64_t>(blockIdx.x) * nt;
  const int64_t iters = first < groups ? (groups - first + span - 1) / span : 0;
  const int64_t full_iters =
      first + nt <= whole ? (iters < (whole - first - nt) / span + 1 ? iters : (whole - first - nt) / span + 1) : 0;
  auto column = [&](int64_t it) { return (first + it * span + tid) * V; };

  Staged<DT, V, R> A, B;
  CeSums<V> cs;
  cs.pg = 0.0;
  double ce = 0.0;
  int64_t it_issue = 0, it_use = 0;
  int st_issue = 0, st_use = 0;
  auto issue = [&](Staged<DT, V, R>& b) {
    planned_issue<DT, V, R, FORM, false>(a, ops, st_issue, column(it_issue), V, b);
    if (++st_issue == steps) {
      st_issue = 0;
      ++it_issue;
    }
  };
  auto use = [&](const Staged<DT, V, R>& b) {
    planned_consume<DT, V, R, FUSED, FORM, false>(a, ops, st_use, column(it_use), V, b, mine, slot_stride, cs);
    if (++st_use == steps) {
#pragma unroll
      for (int c = 0; c < V; ++c) ce += cs.q[c] - cs.s[c] * cs.s[c] * inv_n;
      st_use = 0;
      ++it_use;
    }
  };
  // two super-steps per trip, alternating the operand buffers
  const int64_t total = full_iters * steps;
  if (total > 0) issue(A);
  for (int64_t k = 0; k < total; k += 2) {
    if (k + 1 < total) issue(B);
    use(A);
    if (k + 1 >= total) break;
    if (k + 2 < total) issue(A);
    use(B);
  }
  if (full_iters < iters) {  // the ragged last iteration, not pipelined
    const int64_t col = column(full_iters);
    const int64_t left = a.P - col;
    const int cnt = left >= V ? V : (left > 0 ? static_cast<int>(left) : 0);
    for (int st = 0; st < steps; ++st) {
      planned_issue<DT, V, R, FORM, true>(a, ops, st, col, cnt, A);
      planned_consume<DT, V, R, FUSED, FORM, true>(a, ops, st, col, cnt, A, mine, slot_stride, cs);
    }
#pragma unroll
    for (int c = 0; c < V; ++c)
      if (c < cnt) ce += cs.q[c] - cs.s[c] * cs.s[c] * inv_n;
  }
  double total_ce, total_pg;
  block_sum2(ce, cs.pg, total_ce, total_pg);
  if (tid == 0) {
    a.partials[blockIdx.x] = total_ce;
    a.pg_partials[blockIdx.x] = total_pg;
  }
}

// ---------------------------------------------------------------------------
// a5 standalone: consensus error of the stored x over columns [p_begin, p_end)
// ---------------------------------------------------------------------------

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
// worker 0's value, fp64, workers in order.
template <int DT>
__global__ __launch_bounds__(256) void k_consensus_error(const void* x, int64_t ld, int n,
                                                         int64_t p_begin, int64_t p_end,
                                                         double* partials) {
  constexpr int V = DT == GASLOC_BF16 ? 8 : 4, R = DT == GASLOC_BF16 ? 4 : 8;
  const double inv_n = 1.0 / static_cast<double>(n);
  const int64_t base = p_begin - p_begin % V;
  const int64_t groups = (p_end - base + V - 1) / V;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  double ce = 0.0;
  for (int64_t gi = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; gi < groups; gi += stride) {
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

// a6: network average, fp64 sum in worker order, rounded to the param dtype;
// 16 bytes of columns per thread, the loads of 8 workers in flight at a time.
template <int DT>
__global__ __launch_bounds__(256) void k_replica_mean(const void* x, int64_t ld, int n, int64_t P,
                                                      void* out) {
  constexpr int V = DT == GASLOC_BF16 ? 8 : 4, R = 8;
  const int64_t groups = (P + V - 1) / V;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t gi = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; gi < groups; gi += stride) {
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

template <int DT, int V, bool FUSED, int FORM, typename F>
hipError_t with_planned_typed(F& f) {
  return f(reinterpret_cast<const void*>(&k_gossip_planned<DT, V, kPlanBatch, FUSED, FORM>));
}

template <int DT, bool FUSED, int FORM, typename F>
hipError_t with_planned_vec(const LaunchShape& s, F& f) {
  if (s.vec == 4) return with_planned_typed<DT, 4, FUSED, FORM>(f);
  if (s.vec == 2) return with_planned_typed<DT, 2, FUSED, FORM>(f);
  return with_planned_typed<DT, 1, FUSED, FORM>(f);
}

// As for the phase kernel, the fused last step exists for EQ and ALG1.
template <int DT, typename F>
hipError_t with_planned_dtype(bool fused, int form, const LaunchShape& s, F& f) {
  switch (form) {
    case GASLOC_FORM_ALG1:
      return fused ? with_planned_vec<DT, true, GASLOC_FORM_ALG1>(s, f)
                   : with_planned_vec<DT, false, GASLOC_FORM_ALG1>(s, f);
    case GASLOC_FORM_DADAM:
      return with_planned_vec<DT, false, GASLOC_FORM_DADAM>(s, f);
    case GASLOC_FORM_LOCAL_DADAM:
      return with_planned_vec<DT, false, GASLOC_FORM_LOCAL_DADAM>(s, f);
    default:
      return fused ? with_planned_vec<DT, true, GASLOC_FORM_EQ>(s, f)
                   : with_planned_vec<DT, false, GASLOC_FORM_EQ>(s, f);
  }
}

template <typename F>
hipError_t with_planned_kernel(int dtype, bool fused, int form, const LaunchShape& s, F& f) {
  if (dtype == GASLOC_BF16) return with_planned_dtype<GASLOC_BF16>(fused, form, s, f);
  return with_planned_dtype<GASLOC_F32>(fused, form, s, f);
}

// Launches `kernel` with the round arguments.
hipError_t launch_round_args(const void* kernel, const GossipArgs& a, const LaunchShape& s, size_t lds,
                             hipStream_t stream) {
  GossipArgs arg = a;
  void* args[] = {&arg};
  const hipError_t e = hipLaunchKernel(kernel, dim3(s.blocks), dim3(s.threads), args, lds, stream);
  return e != hipSuccess ? e : hipGetLastError();
}

}  // namespace

size_t gossip_lds_bytes(int n, int nnz, const LaunchShape& s) {
  const size_t z_bytes = static_cast<size_t>(n) * s.threads * s.vec * sizeof(float);
  const size_t rp_bytes = (static_cast<size_t>(n + 1) * sizeof(int32_t) + 7) & ~size_t(7);
  const size_t ent_bytes = static_cast<size_t>(nnz) * sizeof(CsrEntry);
  return z_bytes + rp_bytes + ent_bytes;
}

hipError_t launch_local_adamw(const AdamArgs& a, int dtype, int blocks_per_worker, hipStream_t stream) {
  const dim3 grid(blocks_per_worker, a.n_active);
  if (dtype == GASLOC_BF16)
    hipLaunchKernelGGL((k_local_adamw<GASLOC_BF16>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((k_local_adamw<GASLOC_F32>), grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

size_t planned_lds_bytes(int slots, const LaunchShape& s) {
  return static_cast<size_t>(slots) * s.threads * s.vec * sizeof(float);
}

hipError_t launch_gossip_planned(const GossipArgs& a, int dtype, bool fused, int form, const LaunchShape& s,
                                 hipStream_t stream) {
  auto launch = [&](const void* k) { return launch_round_args(k, a, s, planned_lds_bytes(a.slots, s), stream); };
  return with_planned_kernel(dtype, fused, form, s, launch);
}

hipError_t launch_gossip_round(const GossipArgs& a, int dtype, bool fused, int form, const LaunchShape& s,
                               hipStream_t stream) {
  auto launch = [&](const void* k) { return launch_round_args(k, a, s, gossip_lds_bytes(a.n, a.nnz, s), stream); };
  return with_round_kernel(dtype, fused, form, s, launch);
}

int round_blocks_per_cu(int dtype, bool fused, int form, bool planned, const LaunchShape& s, size_t dyn_lds) {
  int blocks = 0;
  auto occupancy = [&](const void* k) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k, s.threads, dyn_lds);
  };
  const hipError_t e =
      planned ? with_planned_kernel(dtype, fused, form, s, occupancy) : with_round_kernel(dtype, fused, form, s, occupancy);
  return e == hipSuccess ? blocks : 0;
}

hipError_t launch_consensus_error(const void* x, int dtype, int64_t ld, int n, int64_t p_begin,
                                  int64_t p_end, double* partials, int blocks, hipStream_t stream) {
  if (dtype == GASLOC_BF16)
    hipLaunchKernelGGL((k_consensus_error<GASLOC_BF16>), dim3(blocks), dim3(256), 0, stream, x, ld, n,
                       p_begin, p_end, partials);
  else
    hipLaunchKernelGGL((k_consensus_error<GASLOC_F32>), dim3(blocks), dim3(256), 0, stream, x, ld, n,
                       p_begin, p_end, partials);
  return hipGetLastError();
}

hipError_t launch_finalize(const double* partials, int count, double* out, hipStream_t stream) {
  hipLaunchKernelGGL(k_finalize, dim3(1), dim3(256), 0, stream, partials, count, out);
  return hipGetLastError();
}

hipError_t launch_finalize2(const double* a, const double* b, int count, double* out, hipStream_t stream) {
  hipLaunchKernelGGL(k_finalize2, dim3(1), dim3(256), 0, stream, a, b, count, out);
  return hipGetLastError();
}

hipError_t launch_replica_mean(const void* x, int dtype, int64_t ld, int n, int64_t P, void* out,
                               int blocks, hipStream_t stream) {
  if (dtype == GASLOC_BF16)
    hipLaunchKernelGGL((k_replica_mean<GASLOC_BF16>), dim3(blocks), dim3(256), 0, stream, x, ld, n, P,
                       out);
  else
    hipLaunchKernelGGL((k_replica_mean<GASLOC_F32>), dim3(blocks), dim3(256), 0, stream, x, ld, n, P,
                       out);
  return hipGetLastError();
}

}  // namespace gasloc
