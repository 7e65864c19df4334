// Test-only driver for the library's host code under AddressSanitizer and
// UndefinedBehaviorSanitizer (built by tests/test_sanitizers.py with the host
// compiler, no device code): schedule generators, visit planner and its
// verifier (also on corrupted plans), skipped exchanges and the LR schedule,
// on many seeded inputs.  Exits 0 when every check holds.
#include <cstdint>
#include <cstdio>
#include <random>
#include <string>
#include <vector>

#include "internal.h"

extern "C" float gasloc_lr_schedule(float peak, int64_t step, int64_t total_steps, float warmup_frac,
                                    float start_frac, float final_frac);

namespace {

int failures = 0;

void expect(bool ok, const char* what, int n, uint64_t t) {
  if (!ok) {
    std::fprintf(stderr, "FAIL %s (n=%d, t=%llu)\n", what, n, static_cast<unsigned long long>(t));
    ++failures;
  }
}

struct Csr {
  std::vector<int32_t> rp, col;
  std::vector<float> val;
  int32_t nnz = 0;
};

void plan_and_verify(int n, const Csr& w, std::mt19937_64& rng, uint64_t t) {
  for (bool reuse : {false, true}) {
    std::vector<int32_t> ops;
    int slots = 0;
    std::string err;
    const bool ok = gasloc::plan_round(n, w.rp.data(), w.col.data(), w.val.data(), reuse, &ops, &slots, &err);
    expect(ok, "plan_round", n, t);
    if (!ok) continue;
    expect(ops.size() <= gasloc::plan_words_max(n), "plan size bound", n, t);
    // the kernel's form of the plan: slot words scaled to byte offsets
    for (int32_t unit : {4, 1024, 4096}) {
      std::vector<int32_t> scaled = ops;
      expect(gasloc::scale_plan_slots(&scaled, unit, &err), "scale_plan_slots", n, t);
      expect(scaled.size() == ops.size(), "scaled plan size", n, t);
    }
    // corrupted copies must be rejected (or, if a change happens to keep the
    // plan valid, accepted) without reading out of bounds
    for (int trial = 0; trial < 20; ++trial) {
      std::vector<int32_t> bad = ops;
      const size_t k = static_cast<size_t>(rng() % bad.size());
      const int32_t deltas[] = {-1, 1, 7, -1000, 1 << 20};
      bad[k] += deltas[rng() % 5];
      (void)gasloc::verify_plan(n, w.rp.data(), w.col.data(), w.val.data(), reuse, bad.data(),
                                static_cast<int>(bad.size()), slots, &err);
      const int cut = static_cast<int>(rng() % bad.size());
      expect(!gasloc::verify_plan(n, w.rp.data(), w.col.data(), w.val.data(), reuse, ops.data(), cut, slots, &err),
             "truncated plan rejected", n, t);
    }
  }
}

}  // namespace

int main() {
  std::mt19937_64 rng(12345);
  const int kinds[] = {GASLOC_TOPO_RING, GASLOC_TOPO_COMPLETE, GASLOC_TOPO_EXPONENTIAL, GASLOC_TOPO_ONE_PEER_EXP,
                       GASLOC_TOPO_ONE_PEER, GASLOC_TOPO_TWO_PEER, GASLOC_TOPO_RANDOM_REGULAR};
  for (int n : {1, 2, 3, 4, 5, 8, 16, 17, 31, 32, 33, 64}) {
    const int cap = n * n;
    for (int kind : kinds) {
      if (kind == GASLOC_TOPO_RANDOM_REGULAR && (n < 4 || (3 * n) % 2)) continue;
      std::vector<uint8_t> adm(static_cast<size_t>(n) * n, 0);
      for (int i = 0; i < n; ++i)
        for (int j = i + 1; j < n; ++j) adm[static_cast<size_t>(i) * n + j] = adm[static_cast<size_t>(j) * n + i] = rng() % 3 != 0;
      for (bool restricted : {false, true}) {
        if (restricted && kind != GASLOC_TOPO_ONE_PEER && kind != GASLOC_TOPO_TWO_PEER) continue;
        gasloc_topology topo{kind, 3, 7, restricted ? adm.data() : nullptr};
        for (uint64_t t = 0; t < 6; ++t) {
          Csr w;
          w.rp.assign(static_cast<size_t>(n) + 1, 0);
          w.col.assign(static_cast<size_t>(cap), 0);
          w.val.assign(static_cast<size_t>(cap), 0.0f);
          std::string err;
          const bool ok = gasloc::make_topology(topo, n, t, w.rp.data(), w.col.data(), w.val.data(), cap, &w.nnz, &err);
          expect(ok, "make_topology", n, t);
          if (!ok) continue;
          // a too-small output buffer is an error, never an overrun
          if (w.nnz > n) {
            Csr small;
            small.rp.assign(static_cast<size_t>(n) + 1, 0);
            small.col.assign(static_cast<size_t>(w.nnz - 1), 0);
            small.val.assign(static_cast<size_t>(w.nnz - 1), 0.0f);
            expect(!gasloc::make_topology(topo, n, t, small.rp.data(), small.col.data(), small.val.data(), w.nnz - 1,
                                          &small.nnz, &err),
                   "make_topology rejects a short buffer", n, t);
          }
          plan_and_verify(n, w, rng, t);
          // skipped exchanges: random dead workers and failed links
          std::vector<uint8_t> alive(static_cast<size_t>(n)), link(static_cast<size_t>(n) * n);
          for (auto& a : alive) a = rng() % 5 != 0;
          for (auto& l : link) l = rng() % 4 != 0;
          Csr s;
          s.rp.assign(static_cast<size_t>(n) + 1, 0);
          s.col.assign(static_cast<size_t>(cap), 0);
          s.val.assign(static_cast<size_t>(cap), 0.0f);
          const bool sk = gasloc::skip_exchanges(n, w.rp.data(), w.col.data(), w.val.data(), alive.data(), link.data(),
                                                 s.rp.data(), s.col.data(), s.val.data(), cap, &s.nnz, &err);
          expect(sk, "skip_exchanges", n, t);
          if (sk) plan_and_verify(n, s, rng, t);
        }
      }
    }
    // unstructured CSRs: dense rows, missing diagonals, equal rows
    for (int trial = 0; trial < 20; ++trial) {
      Csr w;
      w.rp.assign(1, 0);
      std::vector<int32_t> prev;
      for (int i = 0; i < n; ++i) {
        std::vector<int32_t> cols;
        if (!prev.empty() && rng() % 3 == 0) {
          cols = prev;  // a row equal to the one before it
        } else {
          for (int j = 0; j < n; ++j)
            if (rng() % 4 == 0) cols.push_back(j);
          if (cols.empty()) cols.push_back(static_cast<int32_t>(rng() % n));
        }
        for (int32_t c : cols) {
          w.col.push_back(c);
          w.val.push_back(1.0f / static_cast<float>(cols.size()));
        }
        w.rp.push_back(static_cast<int32_t>(w.col.size()));
        prev = cols;
      }
      w.nnz = static_cast<int32_t>(w.col.size());
      plan_and_verify(n, w, rng, static_cast<uint64_t>(trial));
    }
  }
  for (int64_t s = -2; s < 120; ++s) {
    const float lr = gasloc_lr_schedule(4e-3f, s, 100, 0.1f, 0.01f, 0.0f);
    expect(lr >= 0.0f && lr <= 4e-3f, "lr schedule in range", 0, static_cast<uint64_t>(s + 2));
  }
  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("sanitize_host: ok\n");
  return 0;
}
