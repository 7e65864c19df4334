// Device-side helpers shared by the HIP kernels of the GASLoC round (CDNA4,
// gfx950): parameter storage (fp32, bf16 with round-to-nearest-even),
// streaming loads and stores, fixed-order reductions, the per-element AdamW
// and outer-optimizer updates, and the launch of a round kernel.  Included
// by each kernel file; not installed.
//
// Every kernel streams [n, P] buffers once: the path is HBM-bandwidth bound
// (well under 2 flop per byte), so the kernels use the vector ALU only (no
// MFMA), 16-byte-per-lane loads and stores where the dtype allows, and a
// non-persistent grid whose workgroups take consecutive column tiles in
// dispatch order.
//
// Floating-point contract: no contraction (each product and sum is rounded
// on its own), correctly rounded fp32 division and square root (HIP's
// default), fp64 for every reduction.
#pragma once
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

// 16/8/4-byte register vectors for global memory traffic
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two binary32 values -> two bfloat16 packed in one word (a in the low half),
// round to nearest, ties to even.  gfx950 does this in one instruction
// (v_cvt_pk_bf16_f32), which agrees bit for bit with the integer rounding
// (add 0x7fff plus the kept lsb, keep the top half) on every binary32 value,
// subnormals included, under the kernels' default float mode (fp32
// subnormals preserved); a NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

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
  constexpr int W = (V + 1) / 2;
  uint32_t h[W];
#pragma unroll
  for (int j = 0; j < W; ++j) {
    h[j] = f32x2_to_bf16x2(o[2 * j], 2 * j + 1 < V ? o[2 * j + 1] : 0.0f);
    kept[2 * j] = __uint_as_float(h[j] << 16);
    if (2 * j + 1 < V) kept[2 * j + 1] = __uint_as_float(h[j] & 0xffff0000u);
  }
  if (cnt == V) {
    if constexpr (V == 8) {
      st_stream(reinterpret_cast<u32x4*>(p), u32x4{h[0], h[1], h[2], h[3]});
    } else if constexpr (V == 4) {
      st_stream(reinterpret_cast<u32x2*>(p), u32x2{h[0], h[1]});
    } else if constexpr (V == 2) {
      st_stream(reinterpret_cast<uint32_t*>(p), h[0]);
    } else {
      *p = static_cast<uint16_t>(h[0]);
    }
  } else {
#pragma unroll
    for (int c = 0; c < V; ++c)
      if (c < cnt) p[c] = static_cast<uint16_t>(h[c / 2] >> (16 * (c & 1)));
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
    return __uint_as_float(f32x2_to_bf16x2(v, 0.0f) << 16);
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
// per-element updates: AdamW (a1) and the outer optimizer (a3)
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

__device__ __forceinline__ float outer_step(float base, float d, float& u, float mu, float eta,
                                            int nesterov) {
  u = mu * u + d;
  const float step = nesterov ? d + mu * u : u;
  return base - eta * step;
}

// Launches `kernel` with the round arguments.
inline hipError_t launch_round_args(const void* kernel, const GossipArgs& a, const LaunchShape& s, size_t lds,
                                    hipStream_t stream) {
  GossipArgs arg = a;
  void* args[] = {&arg};
  const hipError_t e = hipLaunchKernel(kernel, dim3(s.blocks), dim3(s.threads), args, lds, stream);
  return e != hipSuccess ? e : hipGetLastError();
}

}  // namespace
}  // namespace gasloc
