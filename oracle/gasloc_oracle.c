/*
 * gasloc_oracle.c -- plain CPU oracle for one GASLoC gossip round.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the slow, obviously-correct reference
 * that the GPU library is checked against.  Only the test suite, the smoke
 * check and the CPU-baseline leg of the benchmark load it; the GPU library
 * never does.  It shares no code, header, table or helper with the library.
 *
 * Paper: "Unifying Local Communications and Local Updates for LLM
 * Pretraining" (GASLoC).  What is computed, and where it is defined:
 *   - inner loop: AdamW steps per worker (Eq. 1 inner loop, Algorithm 1,
 *     App. B "Optimization": decoupled weight decay, betas (0.9, 0.95));
 *   - pseudo-gradient g = x_{t,H} - x_{t,0} (Eq. 1 outer loop);
 *   - outer step x + eta*g, generalised to the Nesterov outer optimizer of
 *     section 4 / App. B "Optimization";
 *   - mixing with W = I - alpha*Lambda (Eq. 1) and the consensus momentum
 *     gamma * [(x_t+eta g_t) - (x_{t-1}+eta g_{t-1})] (Eq. 2, momentum update);
 *   - consensus error ||pi x||^2 = sum_i ||x_i - xbar||^2 (section 3.1,
 *     Notation: pi is the projector onto the disagreement subspace);
 *   - the squared pseudo-gradient norms sum_i ||x_i - y_i||^2 (Eq. 1);
 *   - network average (Algorithm 1 output);
 *   - the round forms of Algorithm 1 and of App. C (DAdam, Local-DAdam), the
 *     learning-rate schedule of App. B and skipped exchanges (section 3.2,
 *     fault tolerance);
 *   - the communication graphs of section 3.2 and App. B.1 (random 1-Peer
 *     matching, random 2-Peer cycle), the static ring and complete graph
 *     of Tables 1-3, and the exponential graphs cited in section 3.2.
 *
 * The file is compiled twice (oracle/build.py):
 *   REAL=float  : arithmetic in fp32, the precision the workloads fix for
 *                 parameters and optimizer state; bf16 parameter storage is
 *                 supported (round-to-nearest-even on every store).
 *   REAL=double (-DORACLE_FP64): arithmetic and state in fp64; parameters stored as fp64.
 * Both builds use -ffp-contract=off: every product and sum is rounded on its
 * own, in the order written here.  Reductions (consensus error, mean) are
 * always fp64.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef ORACLE_FP64
#define REAL double
#define SQRT_REAL sqrt
#else
#define REAL float
#define SQRT_REAL sqrtf
#endif

/* Parameter storage codes understood by this oracle. */
#define ORC_PARAM_NATIVE 0 /* stored as REAL */
#define ORC_PARAM_BF16 1   /* stored as bfloat16 (REAL=float build only) */

int orc_real_size(void) { return (int)sizeof(REAL); }

/* ------------------------------------------------------------------------ */
/* bfloat16: the top 16 bits of an IEEE binary32.                          */
/* ------------------------------------------------------------------------ */

float orc_bf16_to_f32(uint16_t h) {
  uint32_t bits = ((uint32_t)h) << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return f;
}

/* Round-to-nearest-even from binary32 to bfloat16; NaN stays NaN (quiet). */
uint16_t orc_f32_to_bf16(float f) {
  uint32_t bits;
  memcpy(&bits, &f, sizeof bits);
  if ((bits & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((bits >> 16) | 0x0040u);
  uint32_t keep_lsb = (bits >> 16) & 1u;
  bits += 0x7fffu + keep_lsb;
  return (uint16_t)(bits >> 16);
}

static REAL load_param(const void *buf, int dtype, int64_t idx) {
  if (dtype == ORC_PARAM_BF16) return (REAL)orc_bf16_to_f32(((const uint16_t *)buf)[idx]);
  return ((const REAL *)buf)[idx];
}

static void store_param(void *buf, int dtype, int64_t idx, REAL value) {
  if (dtype == ORC_PARAM_BF16)
    ((uint16_t *)buf)[idx] = orc_f32_to_bf16((float)value);
  else
    ((REAL *)buf)[idx] = value;
}

static int dtype_ok(int dtype) {
  if (dtype == ORC_PARAM_NATIVE) return 1;
  return dtype == ORC_PARAM_BF16 && sizeof(REAL) == sizeof(float);
}

/* ------------------------------------------------------------------------ */
/* SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number    */
/* generators", OOPSLA 2014): a Weyl sequence with increment 0x9e3779b97f4a7c15 */
/* passed through the variant-13 64-bit finalizer.                          */
/* ------------------------------------------------------------------------ */

uint64_t orc_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

uint64_t orc_next(uint64_t *state) {
  *state += 0x9e3779b97f4a7c15ULL;
  return orc_mix64(*state);
}

/* The generator state for communication round t: every worker derives the
 * same state from (seed, t), so all of them agree on the round's graph, which
 * App. B.1 redraws for every communication round. */
uint64_t orc_round_state(uint64_t seed, uint64_t t) { return orc_mix64(seed ^ orc_mix64(t)); }

/* Uniform integer in [0, k): reject draws below 2^64 mod k, then reduce. */
uint64_t orc_bounded(uint64_t *state, uint64_t k) {
  uint64_t threshold = (0 - k) % k; /* = 2^64 mod k */
  for (;;) {
    uint64_t r = orc_next(state);
    if (r >= threshold) return r % k;
  }
}

/* Fisher-Yates shuffle: positions N-1 down to 1 swap with a uniform earlier-or-same slot. */
void orc_shuffle(uint64_t *state, int32_t *a, int32_t N) {
  for (int32_t i = N - 1; i >= 1; --i) {
    int32_t j = (int32_t)orc_bounded(state, (uint64_t)i + 1);
    int32_t tmp = a[i];
    a[i] = a[j];
    a[j] = tmp;
  }
}

/* ------------------------------------------------------------------------ */
/* Communication graphs.  Each round's mixing matrix W = I - alpha*Lambda is */
/* row stochastic and every neighbourhood contains the node itself          */
/* (section 3.1, Notation: N_i includes i).  W is built densely in fp64 and */
/* emitted as CSR with ascending columns; weights are rounded once to REAL. */
/* ------------------------------------------------------------------------ */

#define ORC_TOPO_RING 1
#define ORC_TOPO_COMPLETE 2
#define ORC_TOPO_EXPONENTIAL 3
#define ORC_TOPO_ONE_PEER_EXP 4
#define ORC_TOPO_ONE_PEER 5
#define ORC_TOPO_TWO_PEER 6
#define ORC_TOPO_RANDOM_REGULAR 7

#define ORC_MAX_N 64

/* Uniform weights 1/|N_i| over the (deduplicated) neighbourhood: Algorithm 1
 * averages over N_i with weight 1/|N_i|. */
static void uniform_rows(int n, const unsigned char *adj, double *W) {
  for (int i = 0; i < n; ++i) {
    int deg = 0;
    for (int j = 0; j < n; ++j) deg += adj[i * n + j];
    for (int j = 0; j < n; ++j) W[i * n + j] = adj[i * n + j] ? 1.0 / (double)deg : 0.0;
  }
}

/* Number of hops 1, 2, 4, ... strictly below n (= ceil(log2 n)). */
static int exp_hop_count(int n) {
  int count = 0;
  for (int h = 1; h < n; h *= 2) ++count;
  return count;
}

/* Random d-regular simple graph by the configuration (pairing) model:
 * d*n points, point q belongs to node q/d; a uniformly shuffled point list
 * is read in consecutive pairs; a draw with a self-loop or a repeated edge
 * is discarded and a fresh shuffle of the identity is drawn from the same
 * stream.  Returns 0 on success. */
static int random_regular_adj(int n, int d, uint64_t *state, unsigned char *adj) {
  int npts = n * d;
  int32_t *pts = (int32_t *)malloc(sizeof(int32_t) * (size_t)(npts > 0 ? npts : 1));
  if (!pts) return -1;
  for (int attempt = 0; attempt < 100000; ++attempt) {
    memset(adj, 0, (size_t)n * (size_t)n);
    for (int q = 0; q < npts; ++q) pts[q] = q;
    orc_shuffle(state, pts, npts);
    int simple = 1;
    for (int k = 0; k + 1 < npts; k += 2) {
      int a = pts[k] / d, b = pts[k + 1] / d;
      if (a == b || adj[a * n + b]) {
        simple = 0;
        break;
      }
      adj[a * n + b] = 1;
      adj[b * n + a] = 1;
    }
    if (simple) {
      free(pts);
      return 0;
    }
  }
  free(pts);
  return -1;
}

/* Build the mixing matrix of round t into the CSR arrays.  Returns nnz, or
 * -1 on bad arguments / overflow of cap.  `degree` is used by the random
 * regular graph only. */
/* Metropolis-Hastings weights on the graph in adj (self loops ignored):
 * W_ij = 1/(1 + max(d_i, d_j)) for every edge, W_ii = 1 - sum_j W_ij. */
static void metropolis_rows(int n, unsigned char *adj, double *W) {
  int deg[ORC_MAX_N];
  for (int i = 0; i < n; ++i) {
    deg[i] = 0;
    for (int j = 0; j < n; ++j) deg[i] += (j != i && adj[i * n + j]);
  }
  for (int i = 0; i < n; ++i) {
    double off = 0.0;
    for (int j = 0; j < n; ++j) {
      W[i * n + j] = 0.0;
      if (j == i || !adj[i * n + j]) continue;
      int dmax = deg[i] > deg[j] ? deg[i] : deg[j];
      W[i * n + j] = 1.0 / (1.0 + (double)dmax);
      off += W[i * n + j];
    }
    W[i * n + i] = 1.0 - off;
    adj[i * n + i] = 1;
  }
}

/* As orc_topology, with the randomized 1-Peer and 2-Peer selections
 * restricted to the edges of an admissible graph (App. B.1: restrict the
 * possible peer selections to the edges of the underlying graph).
 * admissible: n*n row-major 0/1, symmetric; NULL means the complete graph.
 * A restricted draw keeps a selected pair only if it is admissible, and its
 * weights are Metropolis-Hastings (equal to the uniform 1/2 and 1/3 of the
 * unrestricted draws, and doubly stochastic for any degrees). */
int orc_topology_restricted(int kind, int n, int degree, uint64_t seed, uint64_t t,
                            const unsigned char *admissible, int32_t *row_ptr, int32_t *col, REAL *val,
                            int cap);

int orc_topology(int kind, int n, int degree, uint64_t seed, uint64_t t, int32_t *row_ptr,
                 int32_t *col, REAL *val, int cap) {
  return orc_topology_restricted(kind, n, degree, seed, t, NULL, row_ptr, col, val, cap);
}

int orc_topology_restricted(int kind, int n, int degree, uint64_t seed, uint64_t t,
                            const unsigned char *admissible, int32_t *row_ptr, int32_t *col, REAL *val,
                            int cap) {
  if (n < 1 || n > ORC_MAX_N) return -1;
  unsigned char *adj = (unsigned char *)calloc((size_t)n * (size_t)n, 1);
  double *W = (double *)calloc((size_t)n * (size_t)n, sizeof(double));
  int32_t *sigma = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
  if (!adj || !W || !sigma) {
    free(adj);
    free(W);
    free(sigma);
    return -1;
  }
  int ok = 1;
  uint64_t state = orc_round_state(seed, t);
  for (int i = 0; i < n; ++i) sigma[i] = i;
  if (admissible && kind != ORC_TOPO_ONE_PEER && kind != ORC_TOPO_TWO_PEER) ok = 0;

  if (kind == ORC_TOPO_RING) {
    /* static cycle i-1, i, i+1 (Tables 1-3, "ring") */
    for (int i = 0; i < n; ++i) {
      adj[i * n + i] = 1;
      adj[i * n + (i + 1) % n] = 1;
      adj[i * n + (i + n - 1) % n] = 1;
    }
    uniform_rows(n, adj, W);
  } else if (kind == ORC_TOPO_COMPLETE) {
    /* Lambda = pi: every worker averages all workers (DiLoCo, section 3.1) */
    for (int i = 0; i < n * n; ++i) adj[i] = 1;
    uniform_rows(n, adj, W);
  } else if (kind == ORC_TOPO_EXPONENTIAL) {
    /* static exponential graph: node i receives from i + 1, 2, 4, ... (mod n) */
    for (int i = 0; i < n; ++i) {
      adj[i * n + i] = 1;
      for (int h = 1; h < n; h *= 2) adj[i * n + (i + h) % n] = 1;
    }
    uniform_rows(n, adj, W);
  } else if (kind == ORC_TOPO_ONE_PEER_EXP) {
    /* one-peer exponential graph: round t, node i receives from i + 2^(t mod tau) */
    int tau = exp_hop_count(n);
    for (int i = 0; i < n; ++i) adj[i * n + i] = 1;
    if (tau > 0) {
      int h = 1 << (int)(t % (uint64_t)tau);
      for (int i = 0; i < n; ++i) adj[i * n + (i + h) % n] = 1;
    }
    uniform_rows(n, adj, W);
  } else if (kind == ORC_TOPO_ONE_PEER) {
    /* randomized 1-Peer (section 3.2): a uniform permutation, consecutive
     * entries (sigma(2k), sigma(2k+1)) are paired; an odd node out keeps itself. */
    orc_shuffle(&state, sigma, n);
    for (int i = 0; i < n; ++i) adj[i * n + i] = 1;
    for (int k = 0; 2 * k + 1 < n; ++k) {
      int a = sigma[2 * k], b = sigma[2 * k + 1];
      if (admissible && !admissible[a * n + b]) continue;
      adj[a * n + b] = 1;
      adj[b * n + a] = 1;
    }
    if (admissible)
      metropolis_rows(n, adj, W);
    else
      uniform_rows(n, adj, W);
  } else if (kind == ORC_TOPO_TWO_PEER) {
    /* randomized 2-Peer (section 3.2): the permutation read as a cycle, each
     * node linked with both cyclic neighbours (symmetrised). */
    orc_shuffle(&state, sigma, n);
    for (int i = 0; i < n; ++i) adj[i * n + i] = 1;
    for (int k = 0; k < n; ++k) {
      int a = sigma[k], b = sigma[(k + 1) % n];
      if (admissible && !admissible[a * n + b]) continue;
      adj[a * n + b] = 1;
      adj[b * n + a] = 1;
    }
    if (admissible)
      metropolis_rows(n, adj, W);
    else
      uniform_rows(n, adj, W);
  } else if (kind == ORC_TOPO_RANDOM_REGULAR) {
    /* a fresh random d-regular graph each round, Metropolis-Hastings weights
     * W_ij = 1/(1 + max(deg_i, deg_j)), W_ii = 1 - sum_j W_ij */
    if (degree < 0 || degree >= n || ((int64_t)n * degree) % 2 != 0) {
      ok = 0;
    } else if (random_regular_adj(n, degree, &state, adj) != 0) {
      ok = 0;
    } else {
      int deg[ORC_MAX_N];
      for (int i = 0; i < n; ++i) {
        deg[i] = 0;
        for (int j = 0; j < n; ++j) deg[i] += adj[i * n + j];
      }
      for (int i = 0; i < n; ++i) {
        double off = 0.0;
        for (int j = 0; j < n; ++j) {
          if (j == i || !adj[i * n + j]) continue;
          int dmax = deg[i] > deg[j] ? deg[i] : deg[j];
          W[i * n + j] = 1.0 / (1.0 + (double)dmax);
          off += W[i * n + j];
        }
        W[i * n + i] = 1.0 - off;
        adj[i * n + i] = 1;
      }
    }
  } else {
    ok = 0;
  }

  int nnz = 0;
  if (ok) {
    row_ptr[0] = 0;
    for (int i = 0; i < n && ok; ++i) {
      for (int j = 0; j < n; ++j) {
        if (!adj[i * n + j]) continue;
        if (nnz >= cap) {
          ok = 0;
          break;
        }
        col[nnz] = j;
        val[nnz] = (REAL)W[i * n + j];
        ++nnz;
      }
      row_ptr[i + 1] = nnz;
    }
  }
  free(adj);
  free(W);
  free(sigma);
  return ok ? nnz : -1;
}

/* Fault tolerance (section 3.2, paragraph "Fault tolerance": a round depends
 * only on its activated exchanges, so one that fails may be dropped).  An exchange {i, j}, i != j, is skipped when worker i or j is
 * dead (alive[.] == 0) or the link failed (link_ok[i*n+j] == 0 or
 * link_ok[j*n+i] == 0); each endpoint then keeps for itself the weight it
 * would have given the other: W_ii += W_ij, W_ij = 0.  alive / link_ok may be
 * NULL (all alive / all links up).  The new diagonal is summed in fp64 in
 * ascending column order and rounded once.  Returns the new nnz or -1. */
int orc_skip_exchanges(int n, const int32_t *row_ptr, const int32_t *col, const REAL *val,
                       const unsigned char *alive, const unsigned char *link_ok, int32_t *out_row_ptr,
                       int32_t *out_col, REAL *out_val, int cap) {
  if (n < 1 || n > ORC_MAX_N) return -1;
  double *W = (double *)calloc((size_t)n * (size_t)n, sizeof(double));
  unsigned char *nz = (unsigned char *)calloc((size_t)n * (size_t)n, 1);
  if (!W || !nz) {
    free(W);
    free(nz);
    return -1;
  }
  for (int i = 0; i < n; ++i)
    for (int32_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k) {
      W[i * n + col[k]] = (double)val[k];
      nz[i * n + col[k]] = 1;
    }
  for (int i = 0; i < n; ++i) {
    double diag = W[i * n + i];
    for (int j = 0; j < n; ++j) {
      if (j == i || !nz[i * n + j]) continue;
      int skip = (alive && (!alive[i] || !alive[j])) ||
                 (link_ok && (!link_ok[i * n + j] || !link_ok[j * n + i]));
      if (!skip) continue;
      diag += W[i * n + j];
      W[i * n + j] = 0.0;
      nz[i * n + j] = 0;
    }
    if (diag != W[i * n + i] || nz[i * n + i]) {
      W[i * n + i] = diag;
      nz[i * n + i] = 1;
    }
  }
  int nnz = 0, ok = 1;
  out_row_ptr[0] = 0;
  for (int i = 0; i < n && ok; ++i) {
    for (int j = 0; j < n; ++j) {
      if (!nz[i * n + j]) continue;
      if (nnz >= cap) {
        ok = 0;
        break;
      }
      out_col[nnz] = j;
      out_val[nnz] = (REAL)W[i * n + j];
      ++nnz;
    }
    out_row_ptr[i + 1] = nnz;
  }
  free(W);
  free(nz);
  return ok ? nnz : -1;
}

/* ------------------------------------------------------------------------ */
/* Inner optimizer: AdamW (decoupled weight decay), App. B "Optimization".  */
/* ------------------------------------------------------------------------ */

/* Per-replica scalars for step number k (k >= 1), evaluated in fp64 and
 * rounded once to REAL:
 *   c_wd = 1 - lr*wd,  s1 = lr / (1 - beta1^k),  c2 = sqrt(1 - beta2^k). */
void orc_adamw_scalars(double lr, double beta1, double beta2, double wd, int64_t k, REAL *c_wd,
                       REAL *s1, REAL *c2) {
  *c_wd = (REAL)(1.0 - lr * wd);
  *s1 = (REAL)(lr / (1.0 - pow(beta1, (double)k)));
  *c2 = (REAL)sqrt(1.0 - pow(beta2, (double)k));
}

/* One local AdamW step for every replica i with active[i] != 0.
 *   y : [n, ld] parameters (the live local iterate x_{t,h}), updated in place
 *   g : [n, gld] fp32 gradients of this step
 *   m, v : [n, ld] first and second moments (REAL), updated in place
 *   k : step count of each replica *after* this step (k[i] >= 1 if active)
 * Per element, in this order (two products of each moment update rounded on
 * their own):
 *   w = y*c_wd;  m = b1*m + (1-b1)*g;  v = b2*v + (1-b2)*(g*g);
 *   d = sqrt(v)/c2 + eps;  y = w - s1*(m/d).
 * Returns 0, or -1 on bad arguments. */
int orc_local_step(int n, int64_t P, int64_t ld, int dtype, void *y, const float *g, int64_t gld,
                   REAL *m, REAL *v, const uint8_t *active, const int64_t *k, double lr, double beta1,
                   double beta2, double eps, double wd) {
  if (n < 1 || P < 0 || ld < P || gld < P || !dtype_ok(dtype)) return -1;
  const REAL b1 = (REAL)beta1, b2 = (REAL)beta2;
  const REAL omb1 = (REAL)(1.0 - beta1), omb2 = (REAL)(1.0 - beta2);
  const REAL epsr = (REAL)eps;
  for (int i = 0; i < n; ++i) {
    if (!active[i]) continue;
    if (k[i] < 1) return -1;
    REAL c_wd, s1, c2;
    orc_adamw_scalars(lr, beta1, beta2, wd, k[i], &c_wd, &s1, &c2);
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      REAL gp = (REAL)g[(int64_t)i * gld + p];
      REAL w = load_param(y, dtype, e) * c_wd;
      m[e] = b1 * m[e] + omb1 * gp;
      v[e] = b2 * v[e] + omb2 * (gp * gp);
      REAL d = SQRT_REAL(v[e]) / c2 + epsr;
      w = w - s1 * (m[e] / d);
      store_param(y, dtype, e, w);
    }
  }
  return 0;
}

/* Learning-rate schedule of App. B "Optimization": a warmup over the first
 * warmup_frac of the steps that starts at start_frac of the peak, then
 * cosine decay to final_frac of the peak at the last step.  Linear warmup and
 * a half-cosine are the readings taken for the shapes the paper names.
 *   s < W:  peak * (start + (1 - start) * s / W)
 *   s >= W: peak * (final + (1 - final) * (1 + cos(pi * (s - W) / (T - W))) / 2)
 * with W = floor(warmup_frac * T); evaluated in fp64, returned in fp32. */
float orc_lr_schedule(double peak, int64_t step, int64_t total, double warmup_frac, double start_frac,
                      double final_frac) {
  if (total < 1) return (float)peak;
  if (step < 0) step = 0;
  if (step > total) step = total;
  int64_t W = (int64_t)floor(warmup_frac * (double)total);
  double lr;
  if (step < W) {
    lr = peak * (start_frac + (1.0 - start_frac) * (double)step / (double)W);
  } else if (total == W) {
    lr = peak;
  } else {
    double progress = (double)(step - W) / (double)(total - W);
    double cosine = (1.0 + cos(3.14159265358979323846 * progress)) / 2.0;
    lr = peak * (final_frac + (1.0 - final_frac) * cosine);
  }
  return (float)lr;
}

/* ------------------------------------------------------------------------ */
/* Outer step, mixing and consensus momentum (Eq. 1 outer loop, Eq. 2).    */
/* ------------------------------------------------------------------------ */

/* One gossip round in the form of Eq. 1 / Eq. 2 with a Nesterov (or heavy
 * ball, or plain) outer optimizer.
 *   x  : [n, ld] round anchors x_t (params), overwritten with x_{t+1}
 *   y  : [n, ld] end of the local block y_i = x_{t,H_i}; set to x_{t+1}
 *        afterwards (the next inner loop starts from x_{t+1})
 *   u  : [n, ld] outer momentum (REAL)
 *   zp : [n, ld] previous post-outer iterate x_{t-1} + eta g_{t-1} (REAL);
 *        only used when gamma != 0
 *   z  : [n, ld] scratch (REAL)
 *   row_ptr/col/val : the mixing matrix W of this round (CSR, REAL weights)
 *   rounds_done : rounds completed before this one (the gamma term is
 *        applied from the second round on, "t >= 1" in Eq. 2)
 * Phase 1, every (i, p):  delta = x - y  (= -g, the pseudo-gradient negated);
 *   u = mu*u + delta;  z = x - eta*(delta + mu*u) (Nesterov) or x - eta*u.
 *   With mu = 0 this is z = x + eta*g, the post-local iterate of Eq. 1.
 * Phase 2, every (i, p):  acc = sum_k W_ik z_k in stored column order;
 *   if gamma != 0 and rounds_done > 0: acc = acc + gamma*(z_i - zp_i);
 *   if gamma != 0: zp_i = z_i;  x_i = acc;  y_i = x_i.
 * Returns 0, or -1 on bad arguments. */
int orc_gossip_round(int n, int64_t P, int64_t ld, int dtype, void *x, void *y, REAL *u, REAL *zp,
                     REAL *z, const int32_t *row_ptr, const int32_t *col, const REAL *val,
                     double mu, double eta, int nesterov, double gamma, int64_t rounds_done) {
  if (n < 1 || P < 0 || ld < P || !dtype_ok(dtype)) return -1;
  if (gamma != 0.0 && !zp) return -1;
  if (row_ptr[0] != 0) return -1;
  for (int i = 0; i < n; ++i) {
    if (row_ptr[i + 1] < row_ptr[i]) return -1;
    for (int32_t kk = row_ptr[i]; kk < row_ptr[i + 1]; ++kk)
      if (col[kk] < 0 || col[kk] >= n) return -1;
  }
  const REAL mur = (REAL)mu, etar = (REAL)eta, gammar = (REAL)gamma;

  /* phase 1: pseudo-gradient and outer optimizer step, every worker */
  for (int i = 0; i < n; ++i) {
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      REAL xv = load_param(x, dtype, e);
      REAL yv = load_param(y, dtype, e);
      REAL delta = xv - yv;
      u[e] = mur * u[e] + delta;
      REAL step = nesterov ? delta + mur * u[e] : u[e];
      z[e] = xv - etar * step;
    }
  }

  /* phase 2: neighbour mix of the post-outer iterates plus consensus momentum */
  for (int i = 0; i < n; ++i) {
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      REAL acc = 0;
      for (int32_t kk = row_ptr[i]; kk < row_ptr[i + 1]; ++kk)
        acc = acc + val[kk] * z[(int64_t)col[kk] * ld + p];
      if (gamma != 0.0 && rounds_done > 0) acc = acc + gammar * (z[e] - zp[e]);
      store_param(x, dtype, e, acc);
    }
  }
  if (gamma != 0.0) {
    for (int i = 0; i < n; ++i)
      for (int64_t p = 0; p < P; ++p) zp[(int64_t)i * ld + p] = z[(int64_t)i * ld + p];
  }

  /* the next inner loop starts from the new anchor: x_{t+1,0} = x_{t+1} */
  for (int i = 0; i < n; ++i)
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      store_param(y, dtype, e, load_param(x, dtype, e));
    }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Other round forms.                                                       */
/* ------------------------------------------------------------------------ */

static int csr_ok(int n, const int32_t *row_ptr, const int32_t *col) {
  if (row_ptr[0] != 0) return 0;
  for (int i = 0; i < n; ++i) {
    if (row_ptr[i + 1] < row_ptr[i]) return 0;
    for (int32_t kk = row_ptr[i]; kk < row_ptr[i + 1]; ++kk)
      if (col[kk] < 0 || col[kk] >= n) return 0;
  }
  return 1;
}

/* The outer optimizer step of a worker: momentum u <- mu u + d, then
 * base - eta (d + mu u) (Nesterov) or base - eta u (heavy ball). */
static REAL outer_step(REAL base, REAL d, REAL *u, REAL mur, REAL etar, int nesterov) {
  *u = mur * *u + d;
  REAL step = nesterov ? d + mur * *u : *u;
  return base - etar * step;
}

/* Algorithm 1: every worker feeds the neighbourhood average of
 * (x_i - y_j) to its outer optimizer,
 *   delta_i = sum_k W_ik (x_i - y_{col_k}),  x_i <- OuterOpt(x_i, delta_i),
 * then the next inner loop starts from x_i (y_i = x_i).  No consensus
 * momentum in this form. */
int orc_alg1_round(int n, int64_t P, int64_t ld, int dtype, void *x, void *y, REAL *u,
                   const int32_t *row_ptr, const int32_t *col, const REAL *val, double mu, double eta,
                   int nesterov) {
  if (n < 1 || P < 0 || ld < P || !dtype_ok(dtype) || !csr_ok(n, row_ptr, col)) return -1;
  const REAL mur = (REAL)mu, etar = (REAL)eta;
  for (int i = 0; i < n; ++i) {
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      REAL xi = load_param(x, dtype, e);
      REAL delta = 0;
      for (int32_t kk = row_ptr[i]; kk < row_ptr[i + 1]; ++kk)
        delta = delta + val[kk] * (xi - load_param(y, dtype, (int64_t)col[kk] * ld + p));
      store_param(x, dtype, e, outer_step(xi, delta, &u[e], mur, etar, nesterov));
    }
  }
  /* row i read x_i and the y_j only, so updating x in place above is exact */
  for (int i = 0; i < n; ++i)
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      store_param(y, dtype, e, load_param(x, dtype, e));
    }
  return 0;
}

/* DAdam step (App. C): mix the pre-update parameters and add the local
 * displacement,  x_i <- sum_j w_ij x_j + (y_i - x_i).  z: [n, ld] scratch. */
int orc_dadam_round(int n, int64_t P, int64_t ld, int dtype, void *x, void *y, REAL *z,
                    const int32_t *row_ptr, const int32_t *col, const REAL *val) {
  if (n < 1 || P < 0 || ld < P || !dtype_ok(dtype) || !csr_ok(n, row_ptr, col)) return -1;
  for (int i = 0; i < n; ++i) {
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      REAL acc = 0;
      for (int32_t kk = row_ptr[i]; kk < row_ptr[i + 1]; ++kk)
        acc = acc + val[kk] * load_param(x, dtype, (int64_t)col[kk] * ld + p);
      z[e] = acc + (load_param(y, dtype, e) - load_param(x, dtype, e));
    }
  }
  for (int i = 0; i < n; ++i)
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      store_param(x, dtype, e, z[e]);
      store_param(y, dtype, e, load_param(x, dtype, e));
    }
  return 0;
}

/* Local-DAdam (App. C): the outer optimizer is applied at the end of the
 * local block with a DAdam-style disagreement of the pre-update parameters,
 *   d_i = sum_j w_ij (x_i - x_j),  x_i <- OuterOpt(y_i, d_i).
 * z: [n, ld] scratch. */
int orc_local_dadam_round(int n, int64_t P, int64_t ld, int dtype, void *x, void *y, REAL *u, REAL *z,
                          const int32_t *row_ptr, const int32_t *col, const REAL *val, double mu,
                          double eta, int nesterov) {
  if (n < 1 || P < 0 || ld < P || !dtype_ok(dtype) || !csr_ok(n, row_ptr, col)) return -1;
  const REAL mur = (REAL)mu, etar = (REAL)eta;
  for (int i = 0; i < n; ++i) {
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      REAL xi = load_param(x, dtype, e);
      REAL d = 0;
      for (int32_t kk = row_ptr[i]; kk < row_ptr[i + 1]; ++kk)
        d = d + val[kk] * (xi - load_param(x, dtype, (int64_t)col[kk] * ld + p));
      z[e] = outer_step(load_param(y, dtype, e), d, &u[e], mur, etar, nesterov);
    }
  }
  for (int i = 0; i < n; ++i)
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      store_param(x, dtype, e, z[e]);
      store_param(y, dtype, e, load_param(x, dtype, e));
    }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Consensus error and network average.                                     */
/* ------------------------------------------------------------------------ */

/* ||pi x||^2 = sum_p sum_i (x_ip - xbar_p)^2, xbar_p = (1/n) sum_i x_ip,
 * two passes in fp64 over the stored parameters. */
double orc_consensus_error(int n, int64_t P, int64_t ld, int dtype, const void *x) {
  double total = 0.0;
  for (int64_t p = 0; p < P; ++p) {
    double mean = 0.0;
    for (int i = 0; i < n; ++i) mean += (double)load_param(x, dtype, (int64_t)i * ld + p);
    mean = mean / (double)n;
    for (int i = 0; i < n; ++i) {
      double dev = (double)load_param(x, dtype, (int64_t)i * ld + p) - mean;
      total += dev * dev;
    }
  }
  return total;
}

/* Squared norm of the round's pseudo-gradients, sum_i ||x_i - y_i||^2 (the
 * outer-loop difference of Eq. 1 between the round anchor x_{t,0} and the
 * live local iterate x_{t,H}; y = x for a worker without local steps).  The
 * difference is taken in the working precision, as the round takes it; its
 * square and the sums are fp64. */
double orc_pseudo_gradient_sq(int n, int64_t P, int64_t ld, int dtype, const void *x, const void *y) {
  double total = 0.0;
  for (int i = 0; i < n; ++i)
    for (int64_t p = 0; p < P; ++p) {
      int64_t e = (int64_t)i * ld + p;
      REAL d = load_param(x, dtype, e) - load_param(y, dtype, e);
      total += (double)d * (double)d;
    }
  return total;
}

/* Network average xbar_p = (1/n) sum_i x_ip (Algorithm 1 output), summed in
 * fp64 in replica order, divided in fp64, rounded to the parameter storage. */
void orc_replica_mean(int n, int64_t P, int64_t ld, int dtype, const void *x, void *out) {
  for (int64_t p = 0; p < P; ++p) {
    double s = 0.0;
    for (int i = 0; i < n; ++i) s += (double)load_param(x, dtype, (int64_t)i * ld + p);
    double mean = s / (double)n;
    if (dtype == ORC_PARAM_BF16)
      ((uint16_t *)out)[p] = orc_f32_to_bf16((float)mean);
    else
      ((REAL *)out)[p] = (REAL)mean;
  }
}
