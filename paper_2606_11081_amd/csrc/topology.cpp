// Host-side schedule generation: the mixing matrix W_t of every round.
//
// W = I - alpha * Lambda is row stochastic and each neighbourhood contains
// the worker itself (section 3.1, Notation).  Kinds:
//   ring, complete (Lambda = pi, DiLoCo; section 3.1), the static directed
//   exponential graph and the one-peer exponential graph (cited in section
//   3.2), randomized 1-Peer matching and 2-Peer cycle (section 3.2 and
//   App. B.1: a fresh shared permutation each round), and a random regular
//   graph with Metropolis weights.
// Randomness: SplitMix64 (Steele, Lea & Flood, OOPSLA 2014).
#include <algorithm>
#include <cstdint>
#include <string>
#include <vector>

#include "internal.h"

namespace gasloc {
namespace {

// SplitMix64: state advances by the golden-ratio increment; the output is
// the state passed through the 64-bit finalizer (Stafford's "mix13").
inline uint64_t finalize64(uint64_t v) {
  v ^= v >> 30;
  v *= 0xbf58476d1ce4e5b9ULL;
  v ^= v >> 27;
  v *= 0x94d049bb133111ebULL;
  v ^= v >> 31;
  return v;
}

class SplitMix64 {
 public:
  explicit SplitMix64(uint64_t state) : state_(state) {}
  uint64_t next() {
    state_ += 0x9e3779b97f4a7c15ULL;
    return finalize64(state_);
  }
  // Unbiased integer in [0, bound): draws below 2^64 mod bound are rejected.
  uint64_t below(uint64_t bound) {
    const uint64_t reject_under = (~bound + 1) % bound;
    uint64_t r = next();
    while (r < reject_under) r = next();
    return r % bound;
  }
  // Fisher-Yates over an index vector: slot i (from the top) takes a uniform
  // slot in [0, i].
  void permute(std::vector<int>& a) {
    for (size_t i = a.size(); i-- > 1;) {
      size_t j = static_cast<size_t>(below(static_cast<uint64_t>(i) + 1));
      std::swap(a[i], a[j]);
    }
  }

 private:
  uint64_t state_;
};

std::vector<int> identity(int count) {
  std::vector<int> v(static_cast<size_t>(count));
  for (int i = 0; i < count; ++i) v[static_cast<size_t>(i)] = i;
  return v;
}

// Neighbour sets (always including self), kept sorted and unique.
using Neighbours = std::vector<std::vector<int>>;

Neighbours self_only(int n) {
  Neighbours nb(static_cast<size_t>(n));
  for (int i = 0; i < n; ++i) nb[static_cast<size_t>(i)].push_back(i);
  return nb;
}

void link(Neighbours& nb, int a, int b) {
  nb[static_cast<size_t>(a)].push_back(b);
  nb[static_cast<size_t>(b)].push_back(a);
}

void canonicalize(Neighbours& nb) {
  for (auto& row : nb) {
    std::sort(row.begin(), row.end());
    row.erase(std::unique(row.begin(), row.end()), row.end());
  }
}

// Emits the CSR with uniform weights 1/|N_i| (Algorithm 1 averages its
// neighbourhood), rounded once from fp64 to fp32.
bool emit_uniform(const Neighbours& nb, int32_t* row_ptr, int32_t* col, float* val, int32_t cap,
                  int32_t* nnz, std::string* err) {
  int32_t k = 0;
  row_ptr[0] = 0;
  for (size_t i = 0; i < nb.size(); ++i) {
    const double w = 1.0 / static_cast<double>(nb[i].size());
    for (int j : nb[i]) {
      if (k >= cap) {
        *err = "CSR capacity " + std::to_string(cap) + " too small";
        return false;
      }
      col[k] = j;
      val[k] = static_cast<float>(w);
      ++k;
    }
    row_ptr[i + 1] = k;
  }
  *nnz = k;
  return true;
}

// Emits the CSR with Metropolis-Hastings weights on the neighbour sets:
// 1/(1 + max(d_i, d_j)) off the diagonal (d = neighbours other than self),
// the rest of the row on the diagonal; doubly stochastic for any degrees.
bool emit_metropolis(const Neighbours& nb, int32_t* row_ptr, int32_t* col, float* val, int32_t cap,
                     int32_t* nnz, std::string* err) {
  const int n = static_cast<int>(nb.size());
  int32_t k = 0;
  row_ptr[0] = 0;
  for (int i = 0; i < n; ++i) {
    const auto& row = nb[static_cast<size_t>(i)];
    const int di = static_cast<int>(row.size()) - 1;
    auto weight = [&](int j) {
      const int dj = static_cast<int>(nb[static_cast<size_t>(j)].size()) - 1;
      return 1.0 / (1.0 + static_cast<double>(std::max(di, dj)));
    };
    double off_sum = 0.0;
    for (int j : row)
      if (j != i) off_sum += weight(j);
    for (int j : row) {
      if (k >= cap) {
        *err = "CSR capacity " + std::to_string(cap) + " too small";
        return false;
      }
      col[k] = j;
      val[k] = static_cast<float>(j == i ? 1.0 - off_sum : weight(j));
      ++k;
    }
    row_ptr[i + 1] = k;
  }
  *nnz = k;
  return true;
}

// Random `deg`-regular simple graph: deg*n half-edge points, point q is
// owned by worker q / deg; shuffle, pair consecutive points, retry with a
// fresh shuffle of the identity (same stream) on a loop or repeated edge.
bool sample_regular(int n, int deg, SplitMix64& rng, Neighbours* out) {
  const int points = n * deg;
  std::vector<int> order;
  for (int attempt = 0; attempt < 100000; ++attempt) {
    order = identity(points);
    rng.permute(order);
    Neighbours nb = self_only(n);
    std::vector<uint8_t> taken(static_cast<size_t>(n) * static_cast<size_t>(n), 0);
    bool ok = true;
    for (int q = 0; q + 1 < points; q += 2) {
      const int a = order[static_cast<size_t>(q)] / deg;
      const int b = order[static_cast<size_t>(q) + 1] / deg;
      const size_t ab = static_cast<size_t>(a) * static_cast<size_t>(n) + static_cast<size_t>(b);
      if (a == b || taken[ab]) {
        ok = false;
        break;
      }
      taken[ab] = 1;
      taken[static_cast<size_t>(b) * static_cast<size_t>(n) + static_cast<size_t>(a)] = 1;
      link(nb, a, b);
    }
    if (ok) {
      canonicalize(nb);
      *out = std::move(nb);
      return true;
    }
  }
  return false;
}

}  // namespace

bool make_topology(const gasloc_topology& topo, int n, uint64_t t, int32_t* row_ptr, int32_t* col,
                   float* val, int32_t cap, int32_t* nnz, std::string* err) {
  if (n < 1 || n > kMaxReplicas) {
    *err = "n must be in [1, 64]";
    return false;
  }
  SplitMix64 rng(finalize64(topo.seed ^ finalize64(t)));
  Neighbours nb = self_only(n);
  // App. B.1: the randomized selections may be restricted to the edges of an
  // admissible graph (row-major n*n, symmetric); then weights are Metropolis.
  const uint8_t* adm = topo.admissible;
  if (adm && topo.kind != GASLOC_TOPO_ONE_PEER && topo.kind != GASLOC_TOPO_TWO_PEER) {
    *err = "an admissible graph restricts only the ONE_PEER and TWO_PEER kinds";
    return false;
  }
  auto allowed = [&](int a, int b) {
    return adm == nullptr || adm[static_cast<size_t>(a) * static_cast<size_t>(n) + static_cast<size_t>(b)] != 0;
  };
  switch (topo.kind) {
    case GASLOC_TOPO_RING:
      for (int i = 0; i < n; ++i) link(nb, i, (i + 1) % n);
      break;
    case GASLOC_TOPO_COMPLETE:
      for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) nb[static_cast<size_t>(i)].push_back(j);
      break;
    case GASLOC_TOPO_EXPONENTIAL:
      // directed: row i receives from i + 1, 2, 4, ... (mod n)
      for (int i = 0; i < n; ++i)
        for (int hop = 1; hop < n; hop <<= 1) nb[static_cast<size_t>(i)].push_back((i + hop) % n);
      break;
    case GASLOC_TOPO_ONE_PEER_EXP: {
      int tau = 0;
      while ((1 << tau) < n) ++tau;  // tau = ceil(log2 n)
      if (tau > 0) {
        const int hop = 1 << static_cast<int>(t % static_cast<uint64_t>(tau));
        for (int i = 0; i < n; ++i) nb[static_cast<size_t>(i)].push_back((i + hop) % n);
      }
      break;
    }
    case GASLOC_TOPO_ONE_PEER: {
      std::vector<int> s = identity(n);
      rng.permute(s);
      for (int k = 0; k + 1 < n; k += 2) {
        const int a = s[static_cast<size_t>(k)], b = s[static_cast<size_t>(k) + 1];
        if (allowed(a, b)) link(nb, a, b);
      }
      break;
    }
    case GASLOC_TOPO_TWO_PEER: {
      std::vector<int> s = identity(n);
      rng.permute(s);
      for (int k = 0; k < n; ++k) {
        const int a = s[static_cast<size_t>(k)], b = s[static_cast<size_t>((k + 1) % n)];
        if (allowed(a, b)) link(nb, a, b);
      }
      break;
    }
    case GASLOC_TOPO_RANDOM_REGULAR: {
      const int d = topo.degree;
      if (d < 0 || d >= n || (n * d) % 2 != 0) {
        *err = "random regular graph needs 0 <= degree < n and n*degree even";
        return false;
      }
      if (!sample_regular(n, d, rng, &nb)) {
        *err = "random regular graph: no simple graph after 100000 draws";
        return false;
      }
      return emit_metropolis(nb, row_ptr, col, val, cap, nnz, err);
    }
    default:
      *err = "topology kind " + std::to_string(topo.kind) + " has no generator";
      return false;
  }
  canonicalize(nb);
  if (adm) return emit_metropolis(nb, row_ptr, col, val, cap, nnz, err);
  return emit_uniform(nb, row_ptr, col, val, cap, nnz, err);
}

// Section 3.2, "Fault tolerance": skipped exchanges.  An off-diagonal entry
// (i, j) is removed when worker i or j is dead or the link between them
// failed in either direction; worker i keeps that weight for itself.  The new
// diagonal is the fp64 sum of the old diagonal and the removed weights (in
// ascending column order), rounded once to fp32; a row gets a diagonal entry
// if it had one or if that sum is nonzero.
bool skip_exchanges(int n, const int32_t* rp, const int32_t* col, const float* val, const uint8_t* alive,
                    const uint8_t* link_ok, int32_t* out_rp, int32_t* out_col, float* out_val, int32_t cap,
                    int32_t* nnz, std::string* err) {
  auto keep = [&](int i, int j) {
    if (i == j) return true;
    if (alive && (!alive[i] || !alive[j])) return false;
    const size_t ij = static_cast<size_t>(i) * n + j, ji = static_cast<size_t>(j) * n + i;
    return !(link_ok && (!link_ok[ij] || !link_ok[ji]));
  };
  std::vector<std::pair<int32_t, float>> row;
  int32_t k_out = 0;
  out_rp[0] = 0;
  for (int i = 0; i < n; ++i) {
    double diag = 0.0;
    bool has_diag = false, moved = false;
    float diag_val = 0.0f;
    for (int32_t k = rp[i]; k < rp[i + 1]; ++k)
      if (col[k] == i) {
        diag += static_cast<double>(val[k]);
        diag_val = val[k];
        has_diag = true;
      }
    for (int32_t k = rp[i]; k < rp[i + 1]; ++k)
      if (!keep(i, col[k])) {
        diag += static_cast<double>(val[k]);
        moved = true;
      }
    row.clear();
    for (int32_t k = rp[i]; k < rp[i + 1]; ++k)
      if (col[k] != i && keep(i, col[k])) row.emplace_back(col[k], val[k]);
    if (has_diag || diag != 0.0) {
      const float d = moved ? static_cast<float>(diag) : diag_val;
      row.insert(std::lower_bound(row.begin(), row.end(), std::make_pair(static_cast<int32_t>(i), -1e30f)),
                 std::make_pair(static_cast<int32_t>(i), d));
    }
    if (k_out + static_cast<int32_t>(row.size()) > cap) {
      *err = "CSR capacity " + std::to_string(cap) + " too small";
      return false;
    }
    for (const auto& e : row) {
      out_col[k_out] = e.first;
      out_val[k_out] = e.second;
      ++k_out;
    }
    out_rp[i + 1] = k_out;
  }
  *nnz = k_out;
  return true;
}

}  // namespace gasloc
