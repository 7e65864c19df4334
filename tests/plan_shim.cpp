// Test-only C entry points around the host planner of the slot-reusing
// gossip kernel (paper_2606_11081_amd/csrc/plan.cpp), built by
// tests/test_plan_host.py into a temporary shared library.
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "internal.h"

extern "C" {

// Plans W (CSR, n rows); writes at most cap words to out.  Returns the word
// count, or -1 with the message in err (size err_cap).
int plan_shim_plan(int n, const int32_t* rp, const int32_t* col, const float* val, int reuse_mix, int32_t* out,
                   int cap, int* slots, char* err, int err_cap) {
  std::vector<int32_t> ops;
  std::string e;
  if (!gasloc::plan_round(n, rp, col, val, reuse_mix != 0, &ops, slots, &e)) {
    std::snprintf(err, static_cast<size_t>(err_cap), "%s", e.c_str());
    return -1;
  }
  if (static_cast<int>(ops.size()) > cap) {
    std::snprintf(err, static_cast<size_t>(err_cap), "plan of %zu words exceeds cap %d", ops.size(), cap);
    return -1;
  }
  std::memcpy(out, ops.data(), ops.size() * sizeof(int32_t));
  return static_cast<int>(ops.size());
}

int plan_shim_verify(int n, const int32_t* rp, const int32_t* col, const float* val, int reuse_mix,
                     const int32_t* ops, int len, int slots) {
  std::string e;
  return gasloc::verify_plan(n, rp, col, val, reuse_mix != 0, ops, len, slots, &e) ? 1 : 0;
}

// Scales the slot words of a plan in place (scale_plan_slots); 1 on success.
int plan_shim_scale(int32_t* ops, int len, int32_t unit) {
  std::vector<int32_t> v(ops, ops + len);
  std::string e;
  if (!gasloc::scale_plan_slots(&v, unit, &e)) return 0;
  std::memcpy(ops, v.data(), v.size() * sizeof(int32_t));
  return 1;
}

int plan_shim_reuse_code() { return gasloc::kPlanReuseMix; }

int64_t plan_shim_words_max(int n) { return static_cast<int64_t>(gasloc::plan_words_max(n)); }

int plan_shim_batch() { return gasloc::kPlanBatch; }
int plan_shim_rows() { return gasloc::kPlanRows; }
}
