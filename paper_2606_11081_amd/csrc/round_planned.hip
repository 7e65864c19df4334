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
// before the current one is computed, so the loads of two super-steps are in
// flight together; they are held as raw words and decoded at their use.
// (Super-steps skip the loads they do not need, so the compiler's wait before
// a computation also covers the next super-step's loads; a variant with the
// same accesses on every path, whose waits left them in flight, measured no
// faster.)
//
// Plan words: [S, start_0 .. start_{S-1}], super-step at start_s:
//   npre, nrows, (worker, slot) x npre, row x nrows,
//   then per row: nent, own_slot, (slot, weight bits) x nent, or
//   kPlanReuseMix, own_slot (EQ, DAdam: the previous summed row's sum).
// Slot words arrive as byte offsets (slot * threads * V * 4, scaled on the
// host for the launch), so a slot's LDS address is one add to the thread's
// own base.
#pragma clang fp contract(off)

#include "device_common.h"

namespace gasloc {
namespace {

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

// The value slot of this thread whose plan word (a byte offset) is `off`.
__device__ __forceinline__ float* at_slot(float* mine, int32_t off) {
  return reinterpret_cast<float*>(reinterpret_cast<char*>(mine) + off);
}

template <int DT, int V, int R, bool FUSED, int FORM, bool TAIL>
__device__ __forceinline__ void planned_consume(const GossipArgs& a, plan_word* ops, int st, int64_t p,
                                                int cnt_tail, const Staged<DT, V, R>& b, float* mine,
                                                CeSums<V>& cs) {
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
    float* out = at_slot(mine, slot);
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
      const float* zo = at_slot(mine, ops[pos + 1]);
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
    // rows of exactly four entries (every row of a 3-regular graph with its
    // self-loop) take a branch-free path; the summation order is the same.
    // Only in the EQ form at 2 columns per thread (the many-slot plans such
    // graphs need): elsewhere the extra path costs registers and occupancy
    constexpr bool kFour = kEq && V == 2;
    if (kFour && count == 4) {
      float zk[4][V], wk[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float* src = at_slot(mine, ops[pos + 2 + 2 * t]);
        wk[t] = __int_as_float(ops[pos + 3 + 2 * t]);
#pragma unroll
        for (int c = 0; c < V; ++c) zk[t][c] = src[c];
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int c = 0; c < V; ++c) acc[c] = acc[c] + wk[t] * (kDiff ? xi[c] - zk[t][c] : zk[t][c]);
      }
    } else {
      for (int k0 = 0; k0 < count; k0 += 4) {
        float zk[4][V], wk[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          if (k0 + t >= count) break;
          const float* src = at_slot(mine, ops[pos + 2 + 2 * (k0 + t)]);
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
  float* mine = zs + tid * V;

  // column groups (t0 + it) * nt + tid for the workgroup's steps it < iters
  // (steps t0 .. t0 + iters - 1 of nt groups each): the same count for every
  // thread of the workgroup, so control stays uniform.  Every step but the
  // last one of the whole row gives each thread V columns; in that one,
  // threads past P see cnt < V (0 beyond the end)
  const int64_t groups = (a.P + V - 1) / V;
  const int64_t whole = a.P / V;  // groups with V columns
  const int64_t steps_total = (groups + nt - 1) / nt;
  const int64_t per = a.tile_groups / nt;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * per;
  const int64_t steps_left = steps_total - t0;
  const int64_t iters = steps_left <= 0 ? 0 : (steps_left < per ? steps_left : per);
  const int64_t full_left = whole / nt - t0;  // steps of this workgroup with every thread full
  const int64_t full_iters = full_left <= 0 ? 0 : (full_left < iters ? full_left : iters);
  auto column = [&](int64_t it) { return ((t0 + it) * nt + tid) * V; };

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
    planned_consume<DT, V, R, FUSED, FORM, false>(a, ops, st_use, column(it_use), V, b, mine, cs);
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
      planned_consume<DT, V, R, FUSED, FORM, true>(a, ops, st, col, cnt, A, mine, cs);
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

// Kernel selection, shared by the launcher and the occupancy query: F is
// called with the address of the instantiation that runs.
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

}  // namespace

size_t planned_lds_bytes(int slots, const LaunchShape& s) {
  return static_cast<size_t>(slots) * s.threads * s.vec * sizeof(float);
}

hipError_t launch_gossip_planned(const GossipArgs& a, int dtype, bool fused, int form, const LaunchShape& s,
                                 hipStream_t stream) {
  auto launch = [&](const void* k) { return launch_round_args(k, a, s, planned_lds_bytes(a.slots, s), stream); };
  return with_planned_kernel(dtype, fused, form, s, launch);
}

int planned_blocks_per_cu(int dtype, bool fused, int form, const LaunchShape& s, size_t dyn_lds) {
  int blocks = 0;
  auto occupancy = [&](const void* k) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k, s.threads, dyn_lds);
  };
  return with_planned_kernel(dtype, fused, form, s, occupancy) == hipSuccess ? blocks : 0;
}

}  // namespace gasloc
