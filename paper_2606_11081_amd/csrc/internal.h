// Internal interfaces between the C ABI (runtime.cpp), the schedule
// generator (topology.cpp), the visit planner (plan.cpp) and the HIP kernels
// (adamw.hip, round_phase.hip, round_planned.hip, reductions.hip, with the
// device helpers of device_common.h).  Not installed.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <string>
#include <vector>

#include "gasloc.h"

namespace gasloc {

constexpr int kMaxReplicas = 64;

// Message of the last failing context-free call on this thread (what
// gasloc_last_error(NULL) returns).
void set_thread_error(const std::string& msg);

bool make_topology(const gasloc_topology& topo, int n, uint64_t t, int32_t* row_ptr, int32_t* col,
                   float* val, int32_t cap, int32_t* nnz, std::string* err);
// Visit plan of a round for the slot-reusing kernel (plan.cpp): super-steps
// of at most kPlanBatch new z values and at most kPlanRows rows; the plan is
// checked by verify_plan before it is returned.  With reuse_mix, a row whose
// CSR entries equal those of the row summed just before it is encoded with
// kPlanReuseMix in place of its entry count and takes that row's sum (only
// for round forms whose neighbour sum does not depend on the row itself).
constexpr int kPlanBatch = 4;
constexpr int kPlanRows = 4;
constexpr int32_t kPlanReuseMix = -1;
bool plan_round(int n, const int32_t* rp, const int32_t* col, const float* val, bool reuse_mix,
                std::vector<int32_t>* ops, int* slots_used, std::string* err);
bool verify_plan(int n, const int32_t* rp, const int32_t* col, const float* val, bool reuse_mix,
                 const int32_t* ops, int len, int slots, std::string* err);
// The plan as the kernel reads it: every slot word (new values, each row's
// own slot, each entry's slot) multiplied by `unit`, the byte stride between
// a thread's slots in LDS.  For a plan verify_plan accepted.
bool scale_plan_slots(std::vector<int32_t>* ops, int32_t unit, std::string* err);
// Upper bound on the words of a plan for n workers.
size_t plan_words_max(int n);
bool skip_exchanges(int n, const int32_t* rp, const int32_t* col, const float* val, const uint8_t* alive,
                    const uint8_t* link_ok, int32_t* out_rp, int32_t* out_col, float* out_val, int32_t cap,
                    int32_t* nnz, std::string* err);

// ---------------------------------------------------------------------------
// kernel arguments (passed by value)
// ---------------------------------------------------------------------------

// One local AdamW step over the active workers.  Slot s of the launch works
// on worker rep[s]; bit s of from_x says that worker's live iterate is still
// the round anchor x (first step after a round), so the step reads x.
struct AdamArgs {
  const void* x;
  void* y;
  float* m;
  float* v;
  const float* g;
  int64_t ld, gld, P;
  float c_wd, b1, omb1, b2, omb2, eps;
  int32_t n_active;
  uint64_t from_x;
  int32_t rep[kMaxReplicas];
  float s1[kMaxReplicas];  // lr / (1 - b1^k)
  float c2[kMaxReplicas];  // sqrt(1 - b2^k)
};

// One gossip round; the consensus-error partial of every workgroup goes to
// partials[blockIdx.x], its partial sum of squared pseudo-gradients to
// pg_partials[blockIdx.x].  Workgroup b takes the column groups [b * tile_groups,
// (b + 1) * tile_groups) (a multiple of the workgroup size), in steps of one
// group per thread.
struct GossipArgs {
  void* x;
  const void* y;
  float* u;
  float* zp;
  const int32_t* row_ptr;
  const int32_t* col;
  const float* val;
  double* partials;
  double* pg_partials;
  int64_t ld, P;
  int64_t tile_groups;
  int32_t n, nnz;
  float mu, eta, gamma;
  int32_t nesterov;
  int32_t use_u;        // outer momentum buffer present (mu != 0)
  int32_t apply_gamma;  // gamma term of Eq. 2 (not in the first round)
  int32_t store_zp;     // keep z for the next round's gamma term
  uint64_t stepped;     // bit i: worker i took local steps since the last round

  // planned visit order (k_gossip_planned only): see plan.cpp
  const int32_t* ops;
  int32_t slots;

  // rows that all hold the same entries (k_gossip_shared only): bit j of
  // shared_mask says column j is an entry, with weight shared_w[j]
  uint64_t shared_mask;
  float shared_w[kMaxReplicas];

  // Fused last local step (the fused kernel only): every worker i with bit i
  // of `active` first takes one AdamW step from its live iterate; the new
  // iterate feeds delta directly and is never written back (it is logically
  // reset to the new x by the round).  Scalars are indexed by worker.
  const float* g;
  float* m;
  float* v;
  int64_t gld;
  uint64_t active;
  float c_wd, b1, omb1, b2, omb2, eps;
  float s1[kMaxReplicas];
  float c2[kMaxReplicas];
};

struct LaunchShape {
  int vec;      // columns per thread per step (1, 2 or 4)
  int threads;  // workgroup size
  int blocks;   // workgroups: one per tile of `per` steps of the workgroup
  int batch;    // workers whose loads are issued together (1, 2, 4 or 8)
  int per;      // steps (threads * vec columns each) per workgroup
};

// Launchers: enqueue on `stream`, return the launch status.
hipError_t launch_local_adamw(const AdamArgs& a, int dtype, hipStream_t stream);
hipError_t launch_gossip_round(const GossipArgs& a, int dtype, bool fused, int form,
                               const LaunchShape& shape, hipStream_t stream);
hipError_t launch_gossip_planned(const GossipArgs& a, int dtype, bool fused, int form, const LaunchShape& shape,
                                 hipStream_t stream);
// Rounds whose rows all hold the same entries, EQ form (round_shared.hip):
// shape.vec must be shared_vec(n, dtype); no dynamic LDS.
int shared_vec(int n, int dtype);
hipError_t launch_gossip_shared(const GossipArgs& a, int dtype, bool fused, const LaunchShape& shape,
                                hipStream_t stream);
// Workgroups of the selected phase or planned round kernel that one CU
// holds at once, given its registers, LDS and wave limits (0 if the query
// fails).
int phase_blocks_per_cu(int dtype, bool fused, int form, const LaunchShape& shape, size_t dyn_lds);
int planned_blocks_per_cu(int dtype, bool fused, int form, const LaunchShape& shape, size_t dyn_lds);
// Dynamic LDS bytes of one workgroup of the planned kernel (z slots only).
size_t planned_lds_bytes(int slots, const LaunchShape& shape);
// The standalone consensus error of columns [p_begin, p_end): one partial
// per workgroup of kReduceThreads threads, each taking `per` consecutive
// steps of 16-byte column groups; consensus_error_blocks gives the count.
constexpr int kReduceThreads = 256;
int consensus_error_blocks(int dtype, int64_t p_begin, int64_t p_end, int per);
hipError_t launch_consensus_error(const void* x, int dtype, int64_t ld, int n, int64_t p_begin,
                                  int64_t p_end, int per, double* partials, hipStream_t stream);
hipError_t launch_finalize(const double* partials, int count, double* out, hipStream_t stream);
// out[0] = sum of a[0..count), out[1] = sum of b[0..count), each as launch_finalize sums.
hipError_t launch_finalize2(const double* a, const double* b, int count, double* out, hipStream_t stream);
// The same sums for up to kMaxPartials partials per array, in a fixed order
// that depends only on count: beyond kFinalizeSegment partials, segments of
// kFinalizeSegment consecutive partials are summed first (into seg[0..S) and
// seg[S..2S), S = ceil(count / kFinalizeSegment)), then the segment sums.
constexpr int kFinalizeSegment = 4096;
constexpr int kMaxPartials = 1 << 20;
hipError_t launch_finalize2_large(const double* a, const double* b, int count, double* seg, double* out,
                                  hipStream_t stream);
// *out = the sum of a[0..count), count <= kMaxPartials, in the same
// segmented order (seg: at least ceil(count / kFinalizeSegment) doubles).
hipError_t launch_finalize_large(const double* a, int count, double* seg, double* out, hipStream_t stream);
// The network average of columns [0, P), workgroups as for the consensus error.
hipError_t launch_replica_mean(const void* x, int dtype, int64_t ld, int n, int64_t P, int per, void* out,
                               hipStream_t stream);

// Dynamic LDS bytes one workgroup of the gossip kernel needs (z slots of
// every thread plus the staged CSR); the kernel also uses kStaticLds bytes.
size_t gossip_lds_bytes(int n, int nnz, const LaunchShape& shape);
constexpr size_t kStaticLds = 2 * 1024 / 64 * sizeof(double);

}  // namespace gasloc
