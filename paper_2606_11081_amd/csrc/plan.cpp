// Visit plan of a round for the slot-reusing gossip kernel.
//
// The fused round needs, for each output row i, the post-outer iterates z_j
// of the workers j in row i of W (and z_i itself for the consensus-momentum
// term).  Holding all n of them per column in LDS bounds the columns in
// flight per CU by LDS / (4 n) bytes.  The plan instead emits rows in an order
// that computes each z_j just before its first reader and frees its LDS slot
// after its last reader, so a sparse W needs only a few slots.  Rows are
// grouped into super-steps: the z of up to kPlanBatch workers are computed
// together (their loads in flight at once), then up to kPlanRows rows are
// emitted.  The per-row arithmetic, including the ascending-column summation
// order of every row, is that of the phase kernel; only independent work is
// reordered.
//
// Rows with the same CSR entries (columns and weight bits) have bit-identical
// neighbour sums.  When the round form's sum does not depend on the row itself
// (reuse_mix), such rows follow the first of them directly and take its sum:
// every row of the complete graph, the second row of every 1-Peer pair.  A
// follower must hold its own index among those columns, so its own value is
// live when it is emitted.
//
// Encoding (int32): [S, start_0 .. start_{S-1}], and at start_s super-step s:
//   n_pre, n_rows, (worker, slot) x n_pre, row x n_rows,
//   then per row: n_ent, own_slot, (slot, weight bits) x n_ent,
//   or kPlanReuseMix, own_slot for a row that takes the last summed row's sum
// The planner and its verifier use slot indices; scale_plan_slots turns them
// into the byte offsets the kernel reads, for one launch shape.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "internal.h"

namespace gasloc {

namespace {

bool same_entries(const int32_t* rp, const int32_t* col, const float* val, int a, int b) {
  const int32_t len = rp[a + 1] - rp[a];
  if (rp[b + 1] - rp[b] != len) return false;
  for (int32_t k = 0; k < len; ++k) {
    if (col[rp[a] + k] != col[rp[b] + k]) return false;
    if (std::memcmp(&val[rp[a] + k], &val[rp[b] + k], sizeof(float)) != 0) return false;
  }
  return true;
}

bool has_column(const int32_t* rp, const int32_t* col, int row, int j) {
  return std::binary_search(col + rp[row], col + rp[row + 1], j);
}

// twins[i]: the other rows with row i's CSR entries that hold their own
// index among them, i.e. the rows that can follow i and take its sum.
std::vector<std::vector<int>> find_twins(int n, const int32_t* rp, const int32_t* col, const float* val) {
  std::vector<std::vector<int>> twins(static_cast<size_t>(n));
  std::vector<char> grouped(static_cast<size_t>(n), 0);
  for (int i = 0; i < n; ++i) {
    if (grouped[static_cast<size_t>(i)]) continue;
    std::vector<int> group{i};
    for (int r = i + 1; r < n; ++r)
      if (!grouped[static_cast<size_t>(r)] && same_entries(rp, col, val, i, r)) {
        group.push_back(r);
        grouped[static_cast<size_t>(r)] = 1;
      }
    for (int lead : group)
      for (int r : group)
        if (r != lead && has_column(rp, col, r, r)) twins[static_cast<size_t>(lead)].push_back(r);
  }
  return twins;
}

// One greedy plan starting from row `first`.
void greedy_plan(int n, const int32_t* rp, const int32_t* col, const float* val,
                 const std::vector<std::vector<int>>& twins, int first, std::vector<int32_t>* ops,
                 int* slots_used) {
  constexpr int max_pre = kPlanBatch, max_rows = kPlanRows;
  // need[i]: columns of row i plus i itself, ascending
  std::vector<std::vector<int>> need(static_cast<size_t>(n));
  std::vector<int> uses(static_cast<size_t>(n), 0);
  for (int i = 0; i < n; ++i) {
    auto& nd = need[static_cast<size_t>(i)];
    for (int32_t k = rp[i]; k < rp[i + 1]; ++k) nd.push_back(col[k]);
    nd.push_back(i);
    std::sort(nd.begin(), nd.end());
    nd.erase(std::unique(nd.begin(), nd.end()), nd.end());
    for (int j : nd) ++uses[static_cast<size_t>(j)];
  }
  std::vector<int> slot_of(static_cast<size_t>(n), -1);
  std::vector<char> emitted(static_cast<size_t>(n), 0), follows(static_cast<size_t>(n), 0);
  std::vector<int> free_slots;  // sorted descending: back() is the lowest free slot
  int high = 0, done = 0;
  std::vector<int32_t> body;
  std::vector<int32_t> starts;
  std::vector<int> rows, pres;
  std::vector<int> queue;  // followers still to emit, in order
  size_t queued = 0;
  while (done < n) {
    rows.clear();
    pres.clear();
    for (;;) {
      if (queued < queue.size()) {  // followers go right after their leader
        if (static_cast<int>(rows.size()) >= max_rows) break;
        const int r = queue[queued++];
        rows.push_back(r);
        emitted[static_cast<size_t>(r)] = 1;
        follows[static_cast<size_t>(r)] = 1;
        ++done;
        continue;
      }
      // next row: fewest new z to compute minus slots it frees; ties -> the
      // row with more of its z already live, then the lowest index
      int best = -1, best_cost = 1 << 30, best_new = 0, best_live = -1;
      for (int i = 0; i < n; ++i) {
        if (emitted[static_cast<size_t>(i)]) continue;
        int cost = 0, fresh = 0, live = 0;
        for (int j : need[static_cast<size_t>(i)]) {
          if (slot_of[static_cast<size_t>(j)] < 0) {
            ++cost;
            ++fresh;
          } else {
            ++live;
          }
          if (uses[static_cast<size_t>(j)] == 1) --cost;
        }
        if (done == 0 && rows.empty()) {  // the first row is given
          if (i != first) continue;
          cost = -(1 << 29);
        }
        if (cost < best_cost || (cost == best_cost && live > best_live)) {
          best_cost = cost;
          best = i;
          best_new = fresh;
          best_live = live;
        }
      }
      if (best < 0) break;
      const bool full = static_cast<int>(rows.size()) >= max_rows ||
                        static_cast<int>(pres.size()) + best_new > max_pre;
      if (!rows.empty() && full) break;
      for (int j : need[static_cast<size_t>(best)]) {
        if (slot_of[static_cast<size_t>(j)] >= 0) continue;
        int s;
        if (!free_slots.empty()) {
          s = free_slots.back();
          free_slots.pop_back();
        } else {
          s = high++;
        }
        slot_of[static_cast<size_t>(j)] = s;
        pres.push_back(j);
      }
      rows.push_back(best);
      emitted[static_cast<size_t>(best)] = 1;
      ++done;
      queue.clear();
      queued = 0;
      for (int r : twins[static_cast<size_t>(best)])
        if (!emitted[static_cast<size_t>(r)]) queue.push_back(r);
    }
    // a row that alone needs more than kPlanBatch new z values gets super-steps
    // of its first values with no rows before it
    size_t q = 0;
    while (pres.size() - q > static_cast<size_t>(max_pre)) {
      starts.push_back(static_cast<int32_t>(body.size()));
      body.push_back(max_pre);
      body.push_back(0);
      for (int k = 0; k < max_pre; ++k, ++q) {
        body.push_back(pres[q]);
        body.push_back(slot_of[static_cast<size_t>(pres[q])]);
      }
    }
    starts.push_back(static_cast<int32_t>(body.size()));
    body.push_back(static_cast<int32_t>(pres.size() - q));
    body.push_back(static_cast<int32_t>(rows.size()));
    for (; q < pres.size(); ++q) {
      body.push_back(pres[q]);
      body.push_back(slot_of[static_cast<size_t>(pres[q])]);
    }
    for (int r : rows) body.push_back(r);
    for (int r : rows) {
      if (follows[static_cast<size_t>(r)]) {
        body.push_back(kPlanReuseMix);
        body.push_back(slot_of[static_cast<size_t>(r)]);
        continue;
      }
      body.push_back(rp[r + 1] - rp[r]);
      body.push_back(slot_of[static_cast<size_t>(r)]);
      for (int32_t k = rp[r]; k < rp[r + 1]; ++k) {
        int32_t bits;
        std::memcpy(&bits, &val[k], sizeof bits);
        body.push_back(slot_of[static_cast<size_t>(col[k])]);
        body.push_back(bits);
      }
    }
    // slots are released only after the whole super-step has been emitted
    for (int r : rows)
      for (int j : need[static_cast<size_t>(r)])
        if (--uses[static_cast<size_t>(j)] == 0) free_slots.push_back(slot_of[static_cast<size_t>(j)]);
    std::sort(free_slots.begin(), free_slots.end(), std::greater<int>());
  }
  const int32_t supers = static_cast<int32_t>(starts.size());
  ops->assign(1, supers);
  for (int32_t at : starts) ops->push_back(1 + supers + at);
  ops->insert(ops->end(), body.begin(), body.end());
  *slots_used = high;
}

}  // namespace

size_t plan_words_max(int n) {
  // S <= n + n / kPlanBatch <= 2 n super-steps: 1 + S starts, 2 S counts,
  // 2 n pre words, n row ids, 2 n row headers and 2 nnz <= 2 n^2 entry words
  const size_t m = static_cast<size_t>(n);
  return 1 + 6 * m + 5 * m + 2 * m * m;
}

bool plan_round(int n, const int32_t* rp, const int32_t* col, const float* val, bool reuse_mix,
                std::vector<int32_t>* ops, int* slots_used, std::string* err) {
  const std::vector<std::vector<int>> twins =
      reuse_mix ? find_twins(n, rp, col, val) : std::vector<std::vector<int>>(static_cast<size_t>(n));
  greedy_plan(n, rp, col, val, twins, 0, ops, slots_used);
  // graphs with many live values at once: try a few other first rows and
  // keep the plan that needs the fewest slots (deterministic choice)
  if (*slots_used > 8) {
    std::vector<int32_t> trial;
    int trial_slots = 0;
    const int tries = std::min(n, 8);
    for (int t = 1; t < tries; ++t) {
      greedy_plan(n, rp, col, val, twins, t * n / tries, &trial, &trial_slots);
      if (trial_slots < *slots_used) {
        ops->swap(trial);
        *slots_used = trial_slots;
      }
    }
  }
  return verify_plan(n, rp, col, val, reuse_mix, ops->data(), static_cast<int>(ops->size()), *slots_used, err);
}

// Multiplies every slot word of a verified plan by `unit` (the launch's byte
// stride between slots, so that the kernel adds a word to its own address
// with no multiply): the slot of each new value, each row's own slot and the
// slot of each entry.  Counts, worker and row indices and weights are kept.
bool scale_plan_slots(std::vector<int32_t>* ops, int32_t unit, std::string* err) {
  std::vector<int32_t>& o = *ops;
  const int len = static_cast<int>(o.size());
  if (len < 1 || o[0] < 1 || len < 1 + o[0] || unit < 1) {
    *err = "round plan: cannot scale";
    return false;
  }
  const int supers = o[0];
  int64_t top = 0;
  for (int s = 0; s < supers; ++s) {
    int pc = o[1 + s];
    const int npre = o[pc], nrows = o[pc + 1];
    pc += 2;
    for (int q = 0; q < npre; ++q, pc += 2) {
      top = std::max<int64_t>(top, o[pc + 1]);
      o[pc + 1] *= unit;
    }
    pc += nrows;
    for (int q = 0; q < nrows; ++q) {
      const int nent = o[pc];
      top = std::max<int64_t>(top, o[pc + 1]);
      o[pc + 1] *= unit;
      pc += 2;
      if (nent == kPlanReuseMix) continue;
      for (int e = 0; e < nent; ++e, pc += 2) o[pc] *= unit;
    }
  }
  if ((top + 1) * unit > (int64_t(1) << 30)) {
    *err = "round plan: slot offsets out of range";
    return false;
  }
  return true;
}

// Replays a plan symbolically: the start table points at consecutive
// super-steps that tile the words after it; every slot read holds the worker
// the CSR names; every z is computed exactly once before use; every row is
// emitted exactly once with its CSR entries in order, or (reuse_mix only) as
// taking the sum of the last row summed before it, whose CSR entries it
// shares; slots stay within `slots`; super-steps hold at most kPlanRows rows
// and kPlanBatch new z, and a super-step without rows is followed by one that
// has some.
bool verify_plan(int n, const int32_t* rp, const int32_t* col, const float* val, bool reuse_mix,
                 const int32_t* ops, int len, int slots, std::string* err) {
  auto bad = [&](const char* what) {
    *err = std::string("round plan: ") + what;
    return false;
  };
  if (len < 1 || ops[0] < 1 || ops[0] > 2 * n || len < 1 + ops[0]) return bad("super-step count");
  const int supers = ops[0];
  std::vector<int> holder(static_cast<size_t>(slots), -1);
  std::vector<char> computed(static_cast<size_t>(n), 0), emitted(static_cast<size_t>(n), 0);
  int pc = 1 + supers, rows_seen = 0, last_summed = -1;
  for (int s = 0; s < supers; ++s) {
    if (ops[1 + s] != pc || pc + 2 > len) return bad("super-step start");
    const int npre = ops[pc], nrows = ops[pc + 1];
    pc += 2;
    if (npre < 0 || npre > kPlanBatch || nrows < 0 || nrows > kPlanRows || npre + nrows == 0 ||
        (nrows == 0 && s == supers - 1) || pc + 2 * npre + nrows > len)
      return bad("super-step counts");
    for (int q = 0; q < npre; ++q) {
      const int j = ops[pc++], slot = ops[pc++];
      if (j < 0 || j >= n || computed[static_cast<size_t>(j)] || slot < 0 || slot >= slots) return bad("pre");
      computed[static_cast<size_t>(j)] = 1;
      holder[static_cast<size_t>(slot)] = j;
    }
    const int ids = pc;
    pc += nrows;
    for (int q = 0; q < nrows; ++q) {
      const int r = ops[ids + q];
      if (r < 0 || r >= n || emitted[static_cast<size_t>(r)] || pc + 2 > len) return bad("row id");
      const int nent = ops[pc], own = ops[pc + 1];
      pc += 2;
      if (own < 0 || own >= slots || holder[static_cast<size_t>(own)] != r) return bad("own slot");
      if (nent == kPlanReuseMix) {
        if (!reuse_mix || last_summed < 0 || !same_entries(rp, col, val, last_summed, r)) return bad("reused sum");
        emitted[static_cast<size_t>(r)] = 1;
        ++rows_seen;
        continue;
      }
      if (nent != rp[r + 1] - rp[r] || pc + 2 * nent > len) return bad("row header");
      last_summed = r;
      for (int e = 0; e < nent; ++e) {
        const int slot = ops[pc++];
        int32_t bits;
        std::memcpy(&bits, &val[rp[r] + e], sizeof bits);
        if (slot < 0 || slot >= slots || holder[static_cast<size_t>(slot)] != col[rp[r] + e] || ops[pc++] != bits)
          return bad("entry");
      }
      emitted[static_cast<size_t>(r)] = 1;
      ++rows_seen;
    }
  }
  if (pc != len || rows_seen != n) return bad("trailing data or missing rows");
  return true;
}

}  // namespace gasloc
