// C ABI of libgasloc.so: argument checks, per-context state, scalar
// precompute, CSR staging and kernel launches.  See include/gasloc.h for the
// contract of every call.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <initializer_list>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "gasloc.h"
#include "internal.h"

using gasloc::kMaxReplicas;

namespace {

constexpr int kStageSlots = 4;      // pinned CSR staging slots, reused round-robin
constexpr size_t kPartialWords =
    2 * static_cast<size_t>(gasloc::kMaxPartials) + 2 * (gasloc::kMaxPartials / gasloc::kFinalizeSegment);

thread_local std::string g_thread_error;

std::string format(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return std::string(buf);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t param_bytes(int dtype) { return dtype == GASLOC_BF16 ? 2 : 4; }

// Byte layout of one staged CSR: row_ptr[n+1] | col[n*n] | val[n*n].
size_t csr_stage_bytes(int n) {
  return sizeof(int32_t) * static_cast<size_t>(n + 1) + (sizeof(int32_t) + sizeof(float)) * n * n;
}

// Largest visit plan (plan.cpp) for n workers.
size_t plan_stage_bytes(int n) { return sizeof(int32_t) * gasloc::plan_words_max(n); }

size_t stage_bytes(int n) { return std::max(csr_stage_bytes(n), plan_stage_bytes(n)); }

}  // namespace

void gasloc::set_thread_error(const std::string& msg) { g_thread_error = msg; }

struct gasloc_ctx {
  int n = 0;
  int64_t P = 0;
  gasloc_topology topo{};
  gasloc_hparams hp{};
  gasloc_buffers buf{};
  hipStream_t stream = nullptr;
  int device = 0;
  int cus = 0;

  std::vector<uint8_t> admissible;  // copy of the topology's admissible graph (or empty)
  std::vector<uint8_t> alive;       // 1 per live worker
  bool any_dead = false;
  std::vector<int32_t> skip_rp, skip_col;  // scratch for skipped exchanges
  std::vector<float> skip_val;
  std::vector<int32_t> plan_ops;  // visit plan of the current round
  std::vector<int64_t> k;         // AdamW step count per worker
  std::vector<uint8_t> stepped;   // local steps taken since the last round
  int64_t rounds_done = 0;
  bool ce_current = false;        // d_ce holds the consensus error of the stored x
  bool failed = false;

  unsigned char* d_csr = nullptr;  // device copy of the round's CSR or visit plan
  std::vector<unsigned char> d_csr_key;  // what d_csr holds (kind byte + contents), to skip repeats
  unsigned char* h_stage[kStageSlots] = {};
  hipEvent_t stage_done[kStageSlots] = {};
  bool stage_used[kStageSlots] = {};
  int stage_next = 0;
  // [kPartialWords]: consensus-error partials, pseudo-gradient partials (each
  // kMaxPartials), then the finalize's segment sums
  double* d_partials = nullptr;
  double* d_ce = nullptr;  // [2]: consensus error, squared pseudo-gradients of the last round
  double* h_ce = nullptr;  // [2] pinned

  size_t lds_per_block_max = 0;
  size_t lds_per_cu = 0;

  std::string err;
  // scratch for generated CSRs
  std::vector<int32_t> row_ptr, col;
  std::vector<float> val;
};

namespace {

gasloc_status fail(gasloc_ctx* ctx, gasloc_status st, const std::string& msg) {
  if (ctx) {
    ctx->err = msg;
    if (st == GASLOC_EDEVICE) ctx->failed = true;
  } else {
    g_thread_error = msg;
  }
  return st;
}

gasloc_status hip_fail(gasloc_ctx* ctx, hipError_t e, const char* what) {
  return fail(ctx, GASLOC_EDEVICE, format("%s: %s", what, hipGetErrorString(e)));
}

#define HIP_TRY(ctx, call)                                   \
  do {                                                       \
    hipError_t e_ = (call);                                  \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #call); \
  } while (0)

// Makes ctx->device current for the duration of an ABI call.
class DeviceGuard {
 public:
  explicit DeviceGuard(int device) {
    if (hipGetDevice(&prev_) == hipSuccess && prev_ != device) {
      if (hipSetDevice(device) == hipSuccess) restore_ = true;
    }
  }
  ~DeviceGuard() {
    if (restore_) (void)hipSetDevice(prev_);
  }

 private:
  int prev_ = -1;
  bool restore_ = false;
};

bool finite(float v) { return std::isfinite(v); }

std::string check_hparams(const gasloc_hparams& h) {
  if (!(finite(h.beta1) && h.beta1 >= 0.0f && h.beta1 < 1.0f)) return "beta1 must be in [0, 1)";
  if (!(finite(h.beta2) && h.beta2 >= 0.0f && h.beta2 < 1.0f)) return "beta2 must be in [0, 1)";
  if (!(finite(h.eps) && h.eps > 0.0f)) return "eps must be finite and > 0";
  if (!(finite(h.weight_decay) && h.weight_decay >= 0.0f)) return "weight_decay must be finite and >= 0";
  if (!(finite(h.outer_lr) && h.outer_lr > 0.0f)) return "outer_lr must be finite and > 0";
  if (!(finite(h.outer_momentum) && h.outer_momentum >= 0.0f && h.outer_momentum < 1.0f))
    return "outer_momentum must be in [0, 1)";
  if (h.outer_nesterov != 0 && h.outer_nesterov != 1) return "outer_nesterov must be 0 or 1";
  if (!(finite(h.consensus_momentum) && h.consensus_momentum >= 0.0f && h.consensus_momentum < 1.0f))
    return "consensus_momentum must be in [0, 1)";
  if (h.param_dtype != GASLOC_F32 && h.param_dtype != GASLOC_BF16) return "param_dtype must be F32 or BF16";
  if (h.round_form < GASLOC_FORM_EQ || h.round_form > GASLOC_FORM_LOCAL_DADAM) return "unknown round_form";
  if (h.round_form != GASLOC_FORM_EQ && h.consensus_momentum != 0.0f)
    return "consensus_momentum must be 0 unless round_form is EQ";
  return "";
}

std::string check_csr(const gasloc_csr& W, int n) {
  if (W.n != n) return format("CSR has n=%d, context has n=%d", W.n, n);
  if (!W.row_ptr || (W.nnz > 0 && (!W.col || !W.val))) return "CSR arrays must not be NULL";
  if (W.nnz < n || W.nnz > n * n) return format("CSR nnz=%d outside [n, n*n]", W.nnz);
  if (W.row_ptr[0] != 0 || W.row_ptr[n] != W.nnz) return "CSR row_ptr must start at 0 and end at nnz";
  for (int i = 0; i < n; ++i) {
    const int32_t b = W.row_ptr[i], e = W.row_ptr[i + 1];
    if (e < b || b < 0 || e > W.nnz) return format("CSR row_ptr not monotone at row %d", i);
    double sum = 0.0;
    for (int32_t k = b; k < e; ++k) {
      const int32_t c = W.col[k];
      if (c < 0 || c >= n) return format("CSR column %d out of range in row %d", c, i);
      if (k > b && c <= W.col[k - 1]) return format("CSR columns not strictly ascending in row %d", i);
      if (!std::isfinite(W.val[k])) return format("CSR weight not finite in row %d", i);
      sum += static_cast<double>(W.val[k]);
    }
    if (std::fabs(sum - 1.0) > 1e-6) return format("CSR row %d sums to %.9g, not 1", i, sum);
  }
  return "";
}

// Workgroup shape of the gossip kernel.  The z slots of all n workers live
// in LDS, so LDS bounds the columns in flight per CU; sweeps on the n = 8,
// 16, 32, 64 workloads found 4-column vectors best up to n = 16 and single
// columns (more threads in flight) beyond.  The workgroup is the largest
// whose LDS stays within half a CU's, and loads of 8 workers are batched.
gasloc::LaunchShape pick_gossip_shape(const gasloc_ctx& c, int nnz) {
  const size_t budget = std::min(c.lds_per_cu / 2, c.lds_per_block_max);
  const int widest = c.n <= 16 ? 4 : 1;
  for (int vec : {4, 2, 1}) {
    if (vec > widest) continue;
    for (int threads : {256, 128, 64}) {
      gasloc::LaunchShape s{vec, threads, 0, 8, 0};
      if (gasloc::gossip_lds_bytes(c.n, nnz, s) + gasloc::kStaticLds <= budget) return s;
    }
  }
  return gasloc::LaunchShape{1, 64, 0, 8, 0};
}

// Residency of a round kernel, used to pick the planned kernel's workgroup
// size (the one that keeps the most waves per CU).  It comes from the
// occupancy of the exact kernel that runs (registers, LDS, waves).
//
// LDS is given to a workgroup in granules of 1/128 of the CU's LDS (1280 B
// on MI355X).  The occupancy query counts LDS more finely and over-counts
// LDS-bound residency: measured on the n=32 random 3-regular workload, 128-
// and 64-thread workgroups whose LDS rounds up to one more granule held one
// workgroup fewer than the query said, so the LDS bound is applied here as
// well.
int lds_blocks_per_cu(const gasloc_ctx& c, size_t dyn_lds) {
  const size_t granule = std::max<size_t>(c.lds_per_cu / 128, 1);
  const size_t held = (dyn_lds + gasloc::kStaticLds + granule - 1) / granule * granule;
  return static_cast<int>(c.lds_per_cu / held);
}

// Workgroups of a round kernel resident on one CU at once (at least 1).
int resident_blocks_per_cu(const gasloc_ctx& c, const gasloc::LaunchShape& s, bool fused, bool planned,
                           size_t dyn_lds) {
  const int by_lds = std::min(lds_blocks_per_cu(c, dyn_lds), 2048 / s.threads);
  const int query = planned ? gasloc::planned_blocks_per_cu(c.hp.param_dtype, fused, c.hp.round_form, s, dyn_lds)
                            : gasloc::phase_blocks_per_cu(c.hp.param_dtype, fused, c.hp.round_form, s, dyn_lds);
  return std::max(1, query <= 0 ? by_lds : std::min(query, by_lds));  // a failed query leaves the LDS bound
}

// Grid of a round kernel: the columns are cut into steps of threads * vec
// columns, and workgroup b takes `per` consecutive steps, one after the other,
// then exits.  The grid is not persistent: workgroups are dispatched in column
// order, so the columns in flight form one compact window sweeping the rows
// once (as for the AdamW kernel; a grid-stride loop over a fixed grid spreads
// them over whole rows as its workgroups drift apart).  A few steps per
// workgroup amortise its start (CSR staging, barrier) and its reduction:
// measured on MI355X (gossip round alone), per = 8 against 1 took n=16,
// P=350M from 26.9 to 25.6 ms and n=64, P=50M from 10.7 to 10.4 ms, while 64
// was slower again (26.3, 10.8 ms).  So per = 8, less where that would leave
// fewer than 16 workgroups per CU (n=4, P=1M: 0.031 ms at per = 1, 0.061 at
// 8), and more only if the partials buffer requires it.  The planned kernel
// with more than 8 slots (small LDS-bound workgroups, many of them per CU)
// takes one step per workgroup: on the n=32 random 3-regular bf16 workload
// 1-3% faster than 8 in each of three processes, round alone and fused.
void tile_grid(const gasloc_ctx& c, gasloc::LaunchShape* s, int most_per) {
#ifdef GASLOC_TUNING
  if (const char* env = std::getenv("GASLOC_GOSSIP_PER")) s->per = std::max(0, std::atoi(env));
#endif
  const int64_t groups = (c.P + s->vec - 1) / s->vec;
  const int64_t steps = (groups + s->threads - 1) / s->threads;
  int64_t per = s->per > 0 ? s->per
                           : std::min<int64_t>(most_per, std::max<int64_t>(1, steps / (16 * int64_t(c.cus))));
  per = std::max<int64_t>(per, (steps + gasloc::kMaxPartials - 1) / gasloc::kMaxPartials);
  s->per = static_cast<int>(per);
  s->blocks = static_cast<int>(std::max<int64_t>(1, (steps + per - 1) / per));
}

// Shape override for tuning sweeps, compiled only into a library built with
// -DGASLOC_TUNING: GASLOC_GOSSIP_SHAPE="vec,threads,per,batch" (per 0 =
// computed).  The default build reads no environment here.
void apply_shape_override(gasloc::LaunchShape* s) {
#ifndef GASLOC_TUNING
  (void)s;
#else
  const char* env = std::getenv("GASLOC_GOSSIP_SHAPE");
  if (!env) return;
  int v = 0, t = 0, per = 0, r = 0;
  if (std::sscanf(env, "%d,%d,%d,%d", &v, &t, &per, &r) == 4 && (v == 1 || v == 2 || v == 4) &&
      (t == 64 || t == 128 || t == 256) && per >= 0 && per <= (1 << 20) &&
      (r == 1 || r == 2 || r == 4 || r == 8)) {
    s->vec = v;
    s->threads = t;
    s->per = per;
    s->batch = r;
  }
#endif
}

void release(gasloc_ctx* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  for (int i = 0; i < kStageSlots; ++i) {
    if (c->stage_done[i]) (void)hipEventDestroy(c->stage_done[i]);
    if (c->h_stage[i]) (void)hipHostFree(c->h_stage[i]);
  }
  if (c->h_ce) (void)hipHostFree(c->h_ce);
  if (c->d_csr) (void)hipFree(c->d_csr);
  if (c->d_partials) (void)hipFree(c->d_partials);
  if (c->d_ce) (void)hipFree(c->d_ce);
  delete c;
}

// True if d_csr already holds `parts` (a kind byte, then the contents); else
// records them as what d_csr is about to hold.  A static graph (or plan) is
// then uploaded once, not every round.
using ByteSpan = std::pair<const void*, size_t>;
bool already_uploaded(gasloc_ctx* c, unsigned char kind, std::initializer_list<ByteSpan> parts) {
  size_t len = 1;
  for (const auto& p : parts) len += p.second;
  bool same = c->d_csr_key.size() == len && c->d_csr_key[0] == kind;
  size_t at = 1;
  for (const auto& p : parts) {
    if (!same) break;
    same = std::memcmp(c->d_csr_key.data() + at, p.first, p.second) == 0;
    at += p.second;
  }
  if (same) return true;
  c->d_csr_key.assign(1, kind);
  for (const auto& p : parts) {
    const unsigned char* b = static_cast<const unsigned char*>(p.first);
    c->d_csr_key.insert(c->d_csr_key.end(), b, b + p.second);
  }
  return false;
}

// Copies a CSR into the next pinned slot and enqueues its upload to d_csr
// (nothing if d_csr already holds it).
gasloc_status upload_csr(gasloc_ctx* c, const int32_t* row_ptr, const int32_t* col, const float* val,
                         int nnz) {
  if (already_uploaded(c, 'C', {{row_ptr, sizeof(int32_t) * static_cast<size_t>(c->n + 1)},
                                {col, sizeof(int32_t) * static_cast<size_t>(nnz)},
                                {val, sizeof(float) * static_cast<size_t>(nnz)}}))
    return GASLOC_OK;
  const int slot = c->stage_next;
  c->stage_next = (c->stage_next + 1) % kStageSlots;
  if (c->stage_used[slot]) HIP_TRY(c, hipEventSynchronize(c->stage_done[slot]));
  unsigned char* h = c->h_stage[slot];
  const size_t rp_bytes = sizeof(int32_t) * static_cast<size_t>(c->n + 1);
  const size_t nn = static_cast<size_t>(c->n) * c->n;
  std::memcpy(h, row_ptr, rp_bytes);
  std::memcpy(h + rp_bytes, col, sizeof(int32_t) * static_cast<size_t>(nnz));
  std::memcpy(h + rp_bytes + sizeof(int32_t) * nn, val, sizeof(float) * static_cast<size_t>(nnz));
  HIP_TRY(c, hipMemcpyAsync(c->d_csr, h, csr_stage_bytes(c->n), hipMemcpyHostToDevice, c->stream));
  HIP_TRY(c, hipEventRecord(c->stage_done[slot], c->stream));
  c->stage_used[slot] = true;
  return GASLOC_OK;
}

// Copies a visit plan into the next pinned slot and enqueues its upload
// (nothing if d_csr already holds it).
gasloc_status upload_plan(gasloc_ctx* c, const std::vector<int32_t>& ops) {
  if (sizeof(int32_t) * ops.size() > plan_stage_bytes(c->n))
    return fail(c, GASLOC_EINVAL, "round plan larger than its staging buffer");
  if (already_uploaded(c, 'P', {{ops.data(), sizeof(int32_t) * ops.size()}})) return GASLOC_OK;
  const int slot = c->stage_next;
  c->stage_next = (c->stage_next + 1) % kStageSlots;
  if (c->stage_used[slot]) HIP_TRY(c, hipEventSynchronize(c->stage_done[slot]));
  const size_t bytes = sizeof(int32_t) * ops.size();
  std::memcpy(c->h_stage[slot], ops.data(), bytes);
  HIP_TRY(c, hipMemcpyAsync(c->d_csr, c->h_stage[slot], bytes, hipMemcpyHostToDevice, c->stream));
  HIP_TRY(c, hipEventRecord(c->stage_done[slot], c->stream));
  c->stage_used[slot] = true;
  return GASLOC_OK;
}

// Which kernel runs a round: the phase kernel keeps every worker's slot
// value in LDS; the planned kernel (plan.cpp) keeps only the live ones and
// lets rows with equal entries share one neighbour sum; the shared kernel
// serves rounds whose rows all hold the same entries (the complete graph) in
// the EQ form, with one running sum per column and each row's own term in
// registers.  Measured on MI355X (EQ form, gossip round alone): beyond
// 16 workers planned is faster than phase on every graph (n=64: 1-Peer 15.0 vs
// 28.2 ms, complete 34.5 vs 247 ms; n=32: 3-regular 1.9x, complete 28.8 vs
// 74.8 ms) or tied (n=64 exponential); at n <= 16 the phase kernel keeps more
// loads in flight and the two tie, except the fused round (n=16 one-peer
// exponential: 44.8 vs 45.4 ms) and the complete graph (n=16: 29.8 vs 26.1 ms).
enum class RoundKernel { kPhase, kPlanned, kShared };

// True if every row of W holds the entries of row 0 (columns and weight bits).
bool rows_all_equal(int n, const int32_t* rp, const int32_t* col, const float* val) {
  const int32_t len = rp[1] - rp[0];
  for (int i = 1; i < n; ++i) {
    if (rp[i + 1] - rp[i] != len) return false;
    if (std::memcmp(col + rp[i], col + rp[0], sizeof(int32_t) * static_cast<size_t>(len)) != 0 ||
        std::memcmp(val + rp[i], val + rp[0], sizeof(float) * static_cast<size_t>(len)) != 0)
      return false;
  }
  return true;
}

// The shared kernel on the complete graph (EQ, gamma = 0.1, round alone /
// fused last step + round, against the kernel used before it): fp32 n=16,
// P=350M 25.3-25.7 / 44.3-44.4 ms (planned 25.9-26.0 / 44.3-44.4); n=32,
// P=150M 23.0 / 40.8 ms (planned 28.6 / 45.7); n=64, P=50M 17.8 / 34.1 ms
// (planned 34.8 / 56.6); bf16 n=16 20.6 / 40.9 ms (phase 35.1 / 46.3); n=32
// 23.6 / 46.6 ms (planned 30.9 / 44.6); n=64 22.0 / 34.4 ms (planned 38.1 /
// 55.9).  So it serves every such round except the fused bf16 one at 17-32
// workers.
//
// Test hook (documented in gasloc.h): GASLOC_GOSSIP_KERNEL=phase|planned forces
// one kernel, so that the test suite can run every case through both.
RoundKernel pick_round_kernel(const gasloc_ctx& c, const int32_t* rp, const int32_t* col, const float* val,
                              bool fused) {
  if (const char* env = std::getenv("GASLOC_GOSSIP_KERNEL")) {
    if (std::strcmp(env, "phase") == 0) return RoundKernel::kPhase;
    if (std::strcmp(env, "planned") == 0) return RoundKernel::kPlanned;
  }
  const bool fused_bf16_17_32 = fused && c.hp.param_dtype == GASLOC_BF16 && c.n > 16 && c.n <= 32;
  if (c.hp.round_form == GASLOC_FORM_EQ && !fused_bf16_17_32 && rows_all_equal(c.n, rp, col, val))
    return RoundKernel::kShared;
  return c.n > 16 ? RoundKernel::kPlanned : RoundKernel::kPhase;
}

// Steps of the standalone consensus error per workgroup: 8 (as the round
// kernels), fewer on short ranges so that every CU still gets 16 workgroups.
int reduce_per(const gasloc_ctx& c, int64_t p0, int64_t p1) {
  const int V = c.hp.param_dtype == GASLOC_BF16 ? 8 : 4;
  const int64_t steps = ((p1 - p0 + V) / V + gasloc::kReduceThreads - 1) / gasloc::kReduceThreads;
  return static_cast<int>(std::min<int64_t>(8, std::max<int64_t>(1, steps / (16 * int64_t(c.cus)))));
}

gasloc_status reduce_cols(gasloc_ctx* c, int64_t p0, int64_t p1) {
  const int per = reduce_per(*c, p0, p1);
  const int blocks = gasloc::consensus_error_blocks(c->hp.param_dtype, p0, p1, per);
  HIP_TRY(c, gasloc::launch_consensus_error(c->buf.x, c->hp.param_dtype, c->buf.ld, c->n, p0, p1, per,
                                            c->d_partials, c->stream));
  HIP_TRY(c, gasloc::launch_finalize_large(c->d_partials, blocks, c->d_partials + 2 * gasloc::kMaxPartials,
                                           c->d_ce, c->stream));
  return GASLOC_OK;
}

gasloc_status read_ce(gasloc_ctx* c, double* out) {
  HIP_TRY(c, hipMemcpyAsync(c->h_ce, c->d_ce, sizeof(double), hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  *out = *c->h_ce;
  return GASLOC_OK;
}

// One local AdamW step, planned on the host: the workers it moves and their
// scalars for step number k_i + 1, evaluated in fp64 and rounded once.
struct StepPlan {
  uint64_t active = 0;
  int count = 0;
  float c_wd = 0, b1 = 0, b2 = 0, omb1 = 0, omb2 = 0, eps = 0;
  float s1[kMaxReplicas] = {};
  float c2[kMaxReplicas] = {};
};

gasloc_status check_step(gasloc_ctx* c, const float* grads, int64_t grad_ld, float lr) {
  if (!grads || !aligned16(grads)) return fail(c, GASLOC_EINVAL, "grads must be non-NULL and 16-byte aligned");
  if (grad_ld < c->P || (grad_ld * 4) % 16 != 0)
    return fail(c, GASLOC_EINVAL, "grad_ld must be >= P and a multiple of 4");
  if (!(std::isfinite(lr) && lr >= 0.0f)) return fail(c, GASLOC_EINVAL, "lr must be finite and >= 0");
  return GASLOC_OK;
}

StepPlan plan_step(const gasloc_ctx& c, const uint8_t* active, float lr) {
  StepPlan s;
  const double lr64 = lr, b1 = c.hp.beta1, b2 = c.hp.beta2;
  s.c_wd = static_cast<float>(1.0 - lr64 * static_cast<double>(c.hp.weight_decay));
  s.b1 = c.hp.beta1;
  s.b2 = c.hp.beta2;
  s.omb1 = static_cast<float>(1.0 - b1);
  s.omb2 = static_cast<float>(1.0 - b2);
  s.eps = c.hp.eps;
  for (int i = 0; i < c.n; ++i) {
    if ((active && !active[i]) || !c.alive[static_cast<size_t>(i)]) continue;
    const double k = static_cast<double>(c.k[static_cast<size_t>(i)] + 1);
    s.s1[i] = static_cast<float>(lr64 / (1.0 - std::pow(b1, k)));
    s.c2[i] = static_cast<float>(std::sqrt(1.0 - std::pow(b2, k)));
    s.active |= 1ull << i;
    ++s.count;
  }
  return s;
}

void commit_step(gasloc_ctx* c, const StepPlan& s) {
  for (int i = 0; i < c->n; ++i) {
    if (!((s.active >> i) & 1ull)) continue;
    c->k[static_cast<size_t>(i)] += 1;
    c->stepped[static_cast<size_t>(i)] = 1;
  }
}

// A gossip round, optionally preceded in the same kernel by one local step of
// the workers in `step` (then `grads` holds their gradients).
gasloc_status run_round(gasloc_ctx* c, const gasloc_csr* W, uint64_t t, const StepPlan* step,
                        const float* grads, int64_t grad_ld) {
  const int32_t *rp, *col;
  const float* val;
  int32_t nnz = 0;
  if (W) {
    const std::string e = check_csr(*W, c->n);
    if (!e.empty()) return fail(c, GASLOC_EINVAL, e);
    rp = W->row_ptr;
    col = W->col;
    val = W->val;
    nnz = W->nnz;
  } else {
    if (c->topo.kind == GASLOC_TOPO_EXPLICIT)
      return fail(c, GASLOC_EINVAL, "EXPLICIT topology: pass W to every round");
    std::string err;
    if (!gasloc::make_topology(c->topo, c->n, t, c->row_ptr.data(), c->col.data(), c->val.data(),
                               c->n * c->n, &nnz, &err))
      return fail(c, GASLOC_EINVAL, "topology: " + err);
    rp = c->row_ptr.data();
    col = c->col.data();
    val = c->val.data();
  }
  if (c->any_dead) {
    std::string err;
    if (!gasloc::skip_exchanges(c->n, rp, col, val, c->alive.data(), nullptr, c->skip_rp.data(),
                                c->skip_col.data(), c->skip_val.data(), c->n * c->n, &nnz, &err))
      return fail(c, GASLOC_EINVAL, "skipping exchanges: " + err);
    rp = c->skip_rp.data();
    col = c->skip_col.data();
    val = c->skip_val.data();
  }
  DeviceGuard guard(c->device);
  const RoundKernel kernel = pick_round_kernel(*c, rp, col, val, step != nullptr);
  const bool planned = kernel == RoundKernel::kPlanned;
  int slots = 0;
  if (planned) {
    // rows with equal entries share their neighbour sum where it does not
    // depend on the row (EQ, DAdam)
    const bool reuse_mix = c->hp.round_form == GASLOC_FORM_EQ || c->hp.round_form == GASLOC_FORM_DADAM;
    std::string err;
    if (!gasloc::plan_round(c->n, rp, col, val, reuse_mix, &c->plan_ops, &slots, &err))
      return fail(c, GASLOC_EINVAL, err);
  }
  gasloc::LaunchShape shape;
  size_t lds = 0;
  if (kernel == RoundKernel::kShared) {
    shape = gasloc::LaunchShape{gasloc::shared_vec(c->n, c->hp.param_dtype), 256, 0, 4, 0};
    lds = gasloc::kStaticLds;
  } else if (planned) {
    // 4 columns per thread when the plan needs few slots (n=64 1-Peer: 10.7-
    // 12.8 ms), else 2 (1 column was 25% slower).  The workgroup size is the
    // one that keeps the most waves resident per CU (LDS granules, registers;
    // ties to the larger workgroup): on the n=32 random 3-regular workload,
    // 256 threads for 14-15 slots (5 workgroups, 20 waves, 19.3-19.5 ms) and
    // 128 threads for 16-19 slots (8-9 workgroups, 16-18 waves, 20.5 ms
    // against 21.5-22.0 ms with 4 workgroups of 256).
    shape = gasloc::LaunchShape{slots <= 8 ? 4 : 2, 256, 0, gasloc::kPlanBatch, 0};
    {
      int best_waves = -1;
      gasloc::LaunchShape best = shape;
      for (int vec = shape.vec; vec >= 1 && best_waves < 0; vec /= 2) {
        for (int threads : {256, 128, 64}) {
          gasloc::LaunchShape s{vec, threads, 0, gasloc::kPlanBatch, 0};
          const size_t dyn = gasloc::planned_lds_bytes(slots, s);
          if (dyn + gasloc::kStaticLds > std::min(c->lds_per_cu / 2, c->lds_per_block_max)) continue;
          const int waves = resident_blocks_per_cu(*c, s, step != nullptr, true, dyn) * (threads / 64);
          if (waves > best_waves) {
            best_waves = waves;
            best = s;
          }
        }
      }
      shape = best;
    }
    apply_shape_override(&shape);
    lds = gasloc::planned_lds_bytes(slots, shape) + gasloc::kStaticLds;
  } else {
    shape = pick_gossip_shape(*c, nnz);
    if (step) shape.batch = 4;
    apply_shape_override(&shape);
    if (step && shape.batch == 8) shape.batch = 4;  // the fused kernel batches at most 4 workers
    lds = gasloc::gossip_lds_bytes(c->n, nnz, shape) + gasloc::kStaticLds;
  }
  tile_grid(*c, &shape, planned && slots > 8 ? 1 : 8);
  if (lds > c->lds_per_block_max) return fail(c, GASLOC_EINVAL, "gossip shape exceeds the device's LDS per workgroup");
  if (planned) {  // slot words become byte offsets for this launch's shape
    std::string err;
    if (!gasloc::scale_plan_slots(&c->plan_ops, shape.threads * shape.vec * static_cast<int32_t>(sizeof(float)),
                                  &err))
      return fail(c, GASLOC_EINVAL, err);
  }
  // the shared kernel takes row 0's weights as arguments, not from the device CSR
  if (kernel != RoundKernel::kShared) {
    gasloc_status st = planned ? upload_plan(c, c->plan_ops) : upload_csr(c, rp, col, val, nnz);
    if (st != GASLOC_OK) return st;
  }

  gasloc::GossipArgs a{};
  a.x = c->buf.x;
  a.y = c->buf.y;
  a.u = c->buf.u;
  a.zp = c->buf.zp;
  const size_t rp_bytes = sizeof(int32_t) * static_cast<size_t>(c->n + 1);
  a.row_ptr = reinterpret_cast<const int32_t*>(c->d_csr);
  a.col = reinterpret_cast<const int32_t*>(c->d_csr + rp_bytes);
  a.val = reinterpret_cast<const float*>(c->d_csr + rp_bytes + sizeof(int32_t) * c->n * c->n);
  a.ld = c->buf.ld;
  a.P = c->P;
  a.tile_groups = static_cast<int64_t>(shape.per) * shape.threads;
  a.n = c->n;
  a.nnz = nnz;
  a.mu = c->hp.outer_momentum;
  a.eta = c->hp.outer_lr;
  a.gamma = c->hp.consensus_momentum;
  a.nesterov = c->hp.outer_nesterov;
  a.use_u = c->buf.u != nullptr && c->hp.round_form != GASLOC_FORM_DADAM;
  a.store_zp = c->hp.consensus_momentum != 0.0f;
  a.apply_gamma = a.store_zp && c->rounds_done > 0;
  for (int i = 0; i < c->n; ++i)
    if (c->stepped[static_cast<size_t>(i)]) a.stepped |= (1ull << i);
  if (step) {
    a.g = grads;
    a.gld = grad_ld;
    a.m = c->buf.m;
    a.v = c->buf.v;
    a.active = step->active;
    a.c_wd = step->c_wd;
    a.b1 = step->b1;
    a.b2 = step->b2;
    a.omb1 = step->omb1;
    a.omb2 = step->omb2;
    a.eps = step->eps;
    std::memcpy(a.s1, step->s1, sizeof a.s1);
    std::memcpy(a.c2, step->c2, sizeof a.c2);
  }
  a.partials = c->d_partials;
  a.pg_partials = c->d_partials + gasloc::kMaxPartials;
  if (kernel == RoundKernel::kShared) {
    for (int32_t k = rp[0]; k < rp[1]; ++k) {
      a.shared_mask |= 1ull << col[k];
      a.shared_w[col[k]] = val[k];
    }
    HIP_TRY(c, gasloc::launch_gossip_shared(a, c->hp.param_dtype, step != nullptr, shape, c->stream));
  } else if (planned) {
    a.ops = reinterpret_cast<const int32_t*>(c->d_csr);
    a.slots = slots;
    HIP_TRY(c, gasloc::launch_gossip_planned(a, c->hp.param_dtype, step != nullptr, c->hp.round_form, shape,
                                             c->stream));
  } else {
    HIP_TRY(c, gasloc::launch_gossip_round(a, c->hp.param_dtype, step != nullptr, c->hp.round_form, shape,
                                           c->stream));
  }
  HIP_TRY(c, gasloc::launch_finalize2_large(c->d_partials, a.pg_partials, shape.blocks,
                                             c->d_partials + 2 * gasloc::kMaxPartials, c->d_ce, c->stream));
  if (step) {
    for (int i = 0; i < c->n; ++i)
      if ((step->active >> i) & 1ull) c->k[static_cast<size_t>(i)] += 1;
  }
  c->rounds_done += 1;
  std::fill(c->stepped.begin(), c->stepped.end(), 0);
  c->ce_current = true;
  return GASLOC_OK;
}

}  // namespace

extern "C" {

gasloc_status gasloc_init(int32_t n, int64_t P, const gasloc_topology* topology,
                          const gasloc_hparams* hparams, const gasloc_buffers* buffers, void* hip_stream,
                          gasloc_ctx** out) {
  if (!out) return fail(nullptr, GASLOC_EINVAL, "out must not be NULL");
  *out = nullptr;
  if (!topology || !hparams || !buffers) return fail(nullptr, GASLOC_EINVAL, "NULL argument");
  if (n < 1 || n > kMaxReplicas) return fail(nullptr, GASLOC_EINVAL, format("n=%d outside [1, 64]", n));
  if (P < 1 || P >= (int64_t(1) << 31))
    return fail(nullptr, GASLOC_EINVAL, format("P=%lld outside [1, 2^31)", (long long)P));
  const std::string hp_err = check_hparams(*hparams);
  if (!hp_err.empty()) return fail(nullptr, GASLOC_EINVAL, hp_err);
  const gasloc_buffers& b = *buffers;
  const size_t sp = param_bytes(hparams->param_dtype);
  if (b.ld < P) return fail(nullptr, GASLOC_EINVAL, "ld must be >= P");
  if ((static_cast<uint64_t>(b.ld) * sp) % 16 != 0)
    return fail(nullptr, GASLOC_EINVAL, "ld * sizeof(param) must be a multiple of 16 bytes");
  if (!b.x || !b.y || !b.m || !b.v) return fail(nullptr, GASLOC_EINVAL, "x, y, m, v must not be NULL");
  if (!b.u && hparams->outer_momentum != 0.0f && hparams->round_form != GASLOC_FORM_DADAM)
    return fail(nullptr, GASLOC_EINVAL, "u may be NULL only when outer_momentum == 0");
  if (!b.zp && hparams->consensus_momentum != 0.0f)
    return fail(nullptr, GASLOC_EINVAL, "zp may be NULL only when consensus_momentum == 0");
  const void* const all_buffers[] = {b.x, b.y, b.m, b.v, b.u, b.zp};
  for (const void* p : all_buffers)
    if (p && !aligned16(p)) return fail(nullptr, GASLOC_EINVAL, "buffers must be 16-byte aligned");
  if (topology->kind < GASLOC_TOPO_EXPLICIT || topology->kind > GASLOC_TOPO_RANDOM_REGULAR)
    return fail(nullptr, GASLOC_EINVAL, format("unknown topology kind %d", topology->kind));

  gasloc_ctx* c = new (std::nothrow) gasloc_ctx();
  if (!c) return fail(nullptr, GASLOC_ENOMEM, "context allocation failed");
  c->n = n;
  c->P = P;
  c->topo = *topology;
  c->hp = *hparams;
  c->buf = b;
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->k.assign(static_cast<size_t>(n), 0);
  c->stepped.assign(static_cast<size_t>(n), 0);
  c->alive.assign(static_cast<size_t>(n), 1);
  if (topology->admissible) {
    c->admissible.assign(topology->admissible, topology->admissible + static_cast<size_t>(n) * n);
    auto edge = [&](int i, int j) { return c->admissible[static_cast<size_t>(i) * n + j] != 0; };
    for (int i = 0; i < n; ++i)
      for (int j = 0; j < n; ++j)
        if (edge(i, j) != edge(j, i)) {
          delete c;
          return fail(nullptr, GASLOC_EINVAL, "the admissible graph must be symmetric");
        }
    c->topo.admissible = c->admissible.data();
  }
  c->skip_rp.resize(static_cast<size_t>(n) + 1);
  c->skip_col.resize(static_cast<size_t>(n) * n);
  c->skip_val.resize(static_cast<size_t>(n) * n);
  c->row_ptr.resize(static_cast<size_t>(n) + 1);
  c->col.resize(static_cast<size_t>(n) * n);
  c->val.resize(static_cast<size_t>(n) * n);

  if (c->topo.kind != GASLOC_TOPO_EXPLICIT) {
    int32_t nnz = 0;
    std::string err;
    if (!gasloc::make_topology(c->topo, n, 0, c->row_ptr.data(), c->col.data(), c->val.data(), n * n,
                               &nnz, &err)) {
      delete c;
      return fail(nullptr, GASLOC_EINVAL, "topology: " + err);
    }
  }

  // an allocation that runs out of memory is ENOMEM, any other HIP failure EDEVICE
  auto init_fail = [&](hipError_t e, const char* what) {
    g_thread_error = format("%s: %s", what, hipGetErrorString(e));
    release(c);
    return e == hipErrorOutOfMemory ? GASLOC_ENOMEM : GASLOC_EDEVICE;
  };
  hipError_t e = hipGetDevice(&c->device);
  if (e != hipSuccess) return init_fail(e, "hipGetDevice");
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, c->device);
  if (e != hipSuccess) return init_fail(e, "hipGetDeviceProperties");
  c->cus = std::max(1, prop.multiProcessorCount);
  c->lds_per_block_max = prop.sharedMemPerBlock;
  c->lds_per_cu = prop.maxSharedMemoryPerMultiProcessor > 0 ? prop.maxSharedMemoryPerMultiProcessor
                                                             : prop.sharedMemPerBlock;

  // the densest CSR a round may bring (n*n entries) must still fit one workgroup
  const gasloc::LaunchShape worst = pick_gossip_shape(*c, n * n);
  if (gasloc::gossip_lds_bytes(n, n * n, worst) + gasloc::kStaticLds > c->lds_per_block_max) {
    release(c);
    return fail(nullptr, GASLOC_EINVAL, "gossip workgroup does not fit the device's LDS");
  }

  if ((e = hipMalloc(&c->d_csr, stage_bytes(n))) != hipSuccess) return init_fail(e, "hipMalloc csr");
  if ((e = hipMalloc(&c->d_partials, sizeof(double) * kPartialWords)) != hipSuccess)
    return init_fail(e, "hipMalloc partials");
  if ((e = hipMalloc(&c->d_ce, 2 * sizeof(double))) != hipSuccess) return init_fail(e, "hipMalloc ce");
  if ((e = hipHostMalloc(&c->h_ce, 2 * sizeof(double), hipHostMallocDefault)) != hipSuccess)
    return init_fail(e, "hipHostMalloc ce");
  for (int i = 0; i < kStageSlots; ++i) {
    if ((e = hipHostMalloc(&c->h_stage[i], stage_bytes(n), hipHostMallocDefault)) != hipSuccess)
      return init_fail(e, "hipHostMalloc staging");
    if ((e = hipEventCreateWithFlags(&c->stage_done[i], hipEventDisableTiming)) != hipSuccess)
      return init_fail(e, "hipEventCreate");
  }

  if ((e = hipMemsetAsync(c->d_ce, 0, 2 * sizeof(double), c->stream)) != hipSuccess)
    return init_fail(e, "hipMemsetAsync");
  // zero the optimizer state of every worker, m, v, u, zp: columns [0, P) of
  // each row only (the row padding is the caller's)
  for (float* p : {b.m, b.v, b.u, b.zp}) {
    if (!p) continue;
    if ((e = hipMemset2DAsync(p, sizeof(float) * static_cast<size_t>(b.ld), 0, sizeof(float) * static_cast<size_t>(P),
                              static_cast<size_t>(n), c->stream)) != hipSuccess)
      return init_fail(e, "hipMemset2DAsync");
  }
  *out = c;
  return GASLOC_OK;
}

gasloc_status gasloc_local_step(gasloc_ctx* c, const float* grads, int64_t grad_ld, const uint8_t* active,
                                float lr) {
  if (!c) return fail(nullptr, GASLOC_EINVAL, "NULL context");
  if (c->failed) return fail(c, GASLOC_ESTATE, "context unusable after a device error: " + c->err);
  gasloc_status st = check_step(c, grads, grad_ld, lr);
  if (st != GASLOC_OK) return st;
  DeviceGuard guard(c->device);
  const StepPlan plan = plan_step(*c, active, lr);
  if (plan.count == 0) return GASLOC_OK;

  gasloc::AdamArgs a{};
  a.x = c->buf.x;
  a.y = c->buf.y;
  a.m = c->buf.m;
  a.v = c->buf.v;
  a.g = grads;
  a.ld = c->buf.ld;
  a.gld = grad_ld;
  a.P = c->P;
  a.c_wd = plan.c_wd;
  a.b1 = plan.b1;
  a.b2 = plan.b2;
  a.omb1 = plan.omb1;
  a.omb2 = plan.omb2;
  a.eps = plan.eps;
  int slots = 0;
  for (int i = 0; i < c->n; ++i) {
    if (!((plan.active >> i) & 1ull)) continue;
    a.rep[slots] = i;
    a.s1[slots] = plan.s1[i];
    a.c2[slots] = plan.c2[i];
    if (!c->stepped[static_cast<size_t>(i)]) a.from_x |= (1ull << slots);
    ++slots;
  }
  a.n_active = slots;
  HIP_TRY(c, gasloc::launch_local_adamw(a, c->hp.param_dtype, c->stream));
  commit_step(c, plan);
  return GASLOC_OK;
}

gasloc_status gasloc_gossip_round(gasloc_ctx* c, const gasloc_csr* W, uint64_t t) {
  if (!c) return fail(nullptr, GASLOC_EINVAL, "NULL context");
  if (c->failed) return fail(c, GASLOC_ESTATE, "context unusable after a device error: " + c->err);
  return run_round(c, W, t, nullptr, nullptr, 0);
}

gasloc_status gasloc_local_step_gossip_round(gasloc_ctx* c, const float* grads, int64_t grad_ld,
                                             const uint8_t* active, float lr, const gasloc_csr* W, uint64_t t) {
  if (!c) return fail(nullptr, GASLOC_EINVAL, "NULL context");
  if (c->failed) return fail(c, GASLOC_ESTATE, "context unusable after a device error: " + c->err);
  if (c->hp.round_form == GASLOC_FORM_DADAM || c->hp.round_form == GASLOC_FORM_LOCAL_DADAM)
    return fail(c, GASLOC_EINVAL, "the fused last local step supports the EQ and ALG1 forms");
  gasloc_status st = check_step(c, grads, grad_ld, lr);
  if (st != GASLOC_OK) return st;
  const StepPlan plan = plan_step(*c, active, lr);
  return run_round(c, W, t, plan.count ? &plan : nullptr, grads, grad_ld);
}

gasloc_status gasloc_consensus_error(gasloc_ctx* c, double* out) {
  if (!c || !out) return fail(c, GASLOC_EINVAL, "NULL argument");
  if (c->failed) return fail(c, GASLOC_ESTATE, "context unusable after a device error: " + c->err);
  DeviceGuard guard(c->device);
  if (!c->ce_current) {
    gasloc_status st = reduce_cols(c, 0, c->P);
    if (st != GASLOC_OK) return st;
    c->ce_current = true;
  }
  return read_ce(c, out);
}

gasloc_status gasloc_pseudo_gradient_sq(gasloc_ctx* c, double* out) {
  if (!c || !out) return fail(c, GASLOC_EINVAL, "NULL argument");
  if (c->failed) return fail(c, GASLOC_ESTATE, "context unusable after a device error: " + c->err);
  DeviceGuard guard(c->device);
  HIP_TRY(c, hipMemcpyAsync(c->h_ce + 1, c->d_ce + 1, sizeof(double), hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  *out = c->h_ce[1];
  return GASLOC_OK;
}

gasloc_status gasloc_consensus_error_cols(gasloc_ctx* c, int64_t p_begin, int64_t p_end, double* out) {
  if (!c || !out) return fail(c, GASLOC_EINVAL, "NULL argument");
  if (c->failed) return fail(c, GASLOC_ESTATE, "context unusable after a device error: " + c->err);
  if (p_begin < 0 || p_end < p_begin || p_end > c->P)
    return fail(c, GASLOC_EINVAL, "need 0 <= p_begin <= p_end <= P");
  DeviceGuard guard(c->device);
  gasloc_status st = reduce_cols(c, p_begin, p_end);
  if (st != GASLOC_OK) return st;
  c->ce_current = false;  // d_ce now holds a partial sum
  return read_ce(c, out);
}

gasloc_status gasloc_replica_mean(gasloc_ctx* c, void* out) {
  if (!c) return fail(nullptr, GASLOC_EINVAL, "NULL context");
  if (c->failed) return fail(c, GASLOC_ESTATE, "context unusable after a device error: " + c->err);
  if (!out || !aligned16(out)) return fail(c, GASLOC_EINVAL, "out must be non-NULL and 16-byte aligned");
  DeviceGuard guard(c->device);
  HIP_TRY(c, gasloc::launch_replica_mean(c->buf.x, c->hp.param_dtype, c->buf.ld, c->n, c->P,
                                         reduce_per(*c, 0, c->P), out, c->stream));
  return GASLOC_OK;
}

gasloc_status gasloc_topology_csr(gasloc_ctx* c, uint64_t t, int32_t* row_ptr, int32_t* col, float* val,
                                  int32_t cap, int32_t* nnz) {
  if (!c) return fail(nullptr, GASLOC_EINVAL, "NULL context");
  if (!row_ptr || !col || !val || !nnz) return fail(c, GASLOC_EINVAL, "NULL output array");
  if (c->topo.kind == GASLOC_TOPO_EXPLICIT) return fail(c, GASLOC_EINVAL, "EXPLICIT topology has no generator");
  std::string err;
  if (!gasloc::make_topology(c->topo, c->n, t, row_ptr, col, val, cap, nnz, &err))
    return fail(c, GASLOC_EINVAL, "topology: " + err);
  return GASLOC_OK;
}

gasloc_status gasloc_make_topology(const gasloc_topology* topology, int32_t n, uint64_t t, int32_t* row_ptr,
                                   int32_t* col, float* val, int32_t cap, int32_t* nnz) {
  if (!topology || !row_ptr || !col || !val || !nnz) return fail(nullptr, GASLOC_EINVAL, "NULL argument");
  std::string err;
  if (!gasloc::make_topology(*topology, n, t, row_ptr, col, val, cap, nnz, &err))
    return fail(nullptr, GASLOC_EINVAL, "topology: " + err);
  return GASLOC_OK;
}

gasloc_status gasloc_skip_exchanges(const gasloc_csr* W, const uint8_t* alive, const uint8_t* link_ok,
                                    int32_t* row_ptr, int32_t* col, float* val, int32_t cap, int32_t* nnz) {
  if (!W || !row_ptr || !col || !val || !nnz) return fail(nullptr, GASLOC_EINVAL, "NULL argument");
  if (W->n < 1 || W->n > kMaxReplicas) return fail(nullptr, GASLOC_EINVAL, "n outside [1, 64]");
  const std::string e = check_csr(*W, W->n);
  if (!e.empty()) return fail(nullptr, GASLOC_EINVAL, e);
  std::string err;
  if (!gasloc::skip_exchanges(W->n, W->row_ptr, W->col, W->val, alive, link_ok, row_ptr, col, val, cap, nnz,
                              &err))
    return fail(nullptr, GASLOC_EINVAL, err);
  return GASLOC_OK;
}

gasloc_status gasloc_set_alive(gasloc_ctx* c, const uint8_t* alive) {
  if (!c) return fail(nullptr, GASLOC_EINVAL, "NULL context");
  c->any_dead = false;
  for (int i = 0; i < c->n; ++i) {
    c->alive[static_cast<size_t>(i)] = alive ? (alive[i] ? 1 : 0) : 1;
    if (!c->alive[static_cast<size_t>(i)]) c->any_dead = true;
  }
  return GASLOC_OK;
}

gasloc_status gasloc_validate_csr(const gasloc_csr* W, int32_t n) {
  if (!W) return fail(nullptr, GASLOC_EINVAL, "NULL CSR");
  if (n < 1 || n > kMaxReplicas) return fail(nullptr, GASLOC_EINVAL, "n outside [1, 64]");
  const std::string e = check_csr(*W, n);
  if (!e.empty()) return fail(nullptr, GASLOC_EINVAL, e);
  return GASLOC_OK;
}

gasloc_status gasloc_get_counters(const gasloc_ctx* c, int64_t* k, uint8_t* stepped, int64_t* rounds_done) {
  if (!c) return fail(nullptr, GASLOC_EINVAL, "NULL context");
  for (int i = 0; i < c->n; ++i) {
    if (k) k[i] = c->k[static_cast<size_t>(i)];
    if (stepped) stepped[i] = c->stepped[static_cast<size_t>(i)];
  }
  if (rounds_done) *rounds_done = c->rounds_done;
  return GASLOC_OK;
}

gasloc_status gasloc_set_counters(gasloc_ctx* c, const int64_t* k, const uint8_t* stepped, int64_t rounds_done) {
  if (!c) return fail(nullptr, GASLOC_EINVAL, "NULL context");
  if (rounds_done < 0) return fail(c, GASLOC_EINVAL, "rounds_done must be >= 0");
  if (k)
    for (int i = 0; i < c->n; ++i)
      if (k[i] < 0) return fail(c, GASLOC_EINVAL, "step counts must be >= 0");
  for (int i = 0; i < c->n; ++i) {
    if (k) c->k[static_cast<size_t>(i)] = k[i];
    if (stepped) c->stepped[static_cast<size_t>(i)] = stepped[i] ? 1 : 0;
  }
  c->rounds_done = rounds_done;
  c->ce_current = false;
  return GASLOC_OK;
}

const char* gasloc_last_error(const gasloc_ctx* c) { return c ? c->err.c_str() : g_thread_error.c_str(); }

#ifndef GASLOC_BUILD_INFO
#define GASLOC_BUILD_INFO "sources unknown"
#endif
const char* gasloc_build_info(void) { return GASLOC_BUILD_INFO; }

void gasloc_destroy(gasloc_ctx* c) {
  if (!c) return;
  DeviceGuard guard(c->device);
  release(c);
}

}  // extern "C"
