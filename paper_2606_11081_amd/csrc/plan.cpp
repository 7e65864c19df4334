// Visit plan of a round for the slot-reusing gossip kernel.
//
// The fused round needs, for each output row i, the post-outer iterates z_j
// of the workers j in row i of W (and z_i itself for the consensus-momentum
// term).  Holding all n of them per column in LDS bounds the columns in
// flight per CU by LDS / (4 n) bytes.  The plan instead emits rows in an order
// that computes each z_j just before its first reader and frees its LDS slot
// after its last reader, so a sparse W needs only a few slots.  Rows are
// grouped into super-steps: the z of up to `max_pre` workers are computed
// together (their loads in flight at once), then up to `max_rows` rows are
// emitted.  The per-row arithmetic, including the ascending-column summation
// order of every row, is that of the phase kernel; only independent work is
// reordered.
//
// Encoding (int32): [super-steps] then per super-step
//   n_pre, (worker, slot) x n_pre,
//   n_rows, per row: row, n_ent, (slot, weight bits) x n_ent, own_slot
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "internal.h"

namespace gasloc {

bool plan_round(int n, const int32_t* rp, const int32_t* col, const float* val, int max_pre, int max_rows,
                std::vector<int32_t>* ops, int* slots_used, std::string* err) {
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
  std::vector<char> emitted(static_cast<size_t>(n), 0);
  std::vector<int> free_slots;  // sorted descending: back() is the lowest free slot
  int high = 0, done = 0, supers = 0;
  ops->clear();
  ops->push_back(0);
  std::vector<int> rows, pres;
  while (done < n) {
    rows.clear();
    pres.clear();
    for (;;) {
      // next row: fewest new z to compute minus slots it frees; ties -> lowest index
      int best = -1, best_cost = 1 << 30, best_new = 0;
      for (int i = 0; i < n; ++i) {
        if (emitted[static_cast<size_t>(i)]) continue;
        int cost = 0, fresh = 0;
        for (int j : need[static_cast<size_t>(i)]) {
          if (slot_of[static_cast<size_t>(j)] < 0) {
            ++cost;
            ++fresh;
          }
          if (uses[static_cast<size_t>(j)] == 1) --cost;
        }
        if (cost < best_cost) {
          best_cost = cost;
          best = i;
          best_new = fresh;
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
    }
    ops->push_back(static_cast<int32_t>(pres.size()));
    for (int j : pres) {
      ops->push_back(j);
      ops->push_back(slot_of[static_cast<size_t>(j)]);
    }
    ops->push_back(static_cast<int32_t>(rows.size()));
    for (int r : rows) {
      ops->push_back(r);
      ops->push_back(rp[r + 1] - rp[r]);
      for (int32_t k = rp[r]; k < rp[r + 1]; ++k) {
        int32_t bits;
        std::memcpy(&bits, &val[k], sizeof bits);
        ops->push_back(slot_of[static_cast<size_t>(col[k])]);
        ops->push_back(bits);
      }
      ops->push_back(slot_of[static_cast<size_t>(r)]);
    }
    // slots are released only after the whole super-step has been emitted
    for (int r : rows)
      for (int j : need[static_cast<size_t>(r)])
        if (--uses[static_cast<size_t>(j)] == 0) free_slots.push_back(slot_of[static_cast<size_t>(j)]);
    std::sort(free_slots.begin(), free_slots.end(), std::greater<int>());
    ++supers;
  }
  (*ops)[0] = supers;
  *slots_used = high;
  return verify_plan(n, rp, col, val, ops->data(), static_cast<int>(ops->size()), high, max_rows, err);
}

// Replays a plan symbolically: every slot read holds the worker the CSR
// names, every z is computed exactly once before use, every row is emitted
// exactly once with its CSR entries in order, slots stay within `slots`,
// super-steps hold at most max_rows rows.
bool verify_plan(int n, const int32_t* rp, const int32_t* col, const float* val, const int32_t* ops, int len,
                 int slots, int max_rows, std::string* err) {
  auto bad = [&](const char* what) {
    *err = std::string("round plan: ") + what;
    return false;
  };
  if (len < 1 || ops[0] < 1 || ops[0] > n) return bad("super-step count");
  std::vector<int> holder(static_cast<size_t>(slots), -1);
  std::vector<char> computed(static_cast<size_t>(n), 0), emitted(static_cast<size_t>(n), 0);
  int pc = 1, rows_seen = 0;
  for (int s = 0; s < ops[0]; ++s) {
    if (pc >= len) return bad("truncated");
    const int npre = ops[pc++];
    if (npre < 0 || pc + 2 * npre + 1 > len) return bad("pre count");
    for (int q = 0; q < npre; ++q) {
      const int j = ops[pc++], slot = ops[pc++];
      if (j < 0 || j >= n || computed[static_cast<size_t>(j)] || slot < 0 || slot >= slots) return bad("pre");
      computed[static_cast<size_t>(j)] = 1;
      holder[static_cast<size_t>(slot)] = j;
    }
    const int nrows = ops[pc++];
    if (nrows < 1 || nrows > max_rows) return bad("row count");
    for (int q = 0; q < nrows; ++q) {
      if (pc + 2 > len) return bad("truncated row");
      const int r = ops[pc++], nent = ops[pc++];
      if (r < 0 || r >= n || emitted[static_cast<size_t>(r)] || nent != rp[r + 1] - rp[r] ||
          pc + 2 * nent + 1 > len)
        return bad("row header");
      for (int e = 0; e < nent; ++e) {
        const int slot = ops[pc++];
        int32_t bits;
        std::memcpy(&bits, &val[rp[r] + e], sizeof bits);
        if (slot < 0 || slot >= slots || holder[static_cast<size_t>(slot)] != col[rp[r] + e] ||
            ops[pc++] != bits)
          return bad("entry");
      }
      const int own = ops[pc++];
      if (own < 0 || own >= slots || holder[static_cast<size_t>(own)] != r) return bad("own slot");
      emitted[static_cast<size_t>(r)] = 1;
      ++rows_seen;
    }
  }
  if (pc != len || rows_seen != n) return bad("trailing data or missing rows");
  return true;
}

}  // namespace gasloc
