/*
 * gasloc.h -- C ABI of libgasloc.so: one GASLoC gossip round over n worker
 * replicas held on a single AMD MI355X (gfx950) as flat [n, P] buffers.
 *
 * Paper: "Unifying Local Communications and Local Updates for LLM
 * Pretraining" (GASLoC).  A round is
 *   (1) H_i local AdamW steps per worker      (Eq. 1 inner loop, Algorithm 1,
 *                                               App. B "Optimization")
 *   (2) the pseudo-gradient g = x_{t,H} - x_{t,0}            (Eq. 1 outer loop)
 *   (3) the outer Nesterov step, the neighbour mix x <- W z and the consensus
 *       momentum gamma * (z_t - z_{t-1})      (Eq. 1, Eq. 2 "momentum update";
 *                                               Nesterov: section 4, App. B)
 *   (4) the consensus error sum_i ||x_i - xbar||^2    (section 3.1, Notation)
 *
 * Conventions shared by every call:
 *   - Status codes are returned, never thrown; gasloc_last_error() gives the
 *     message of the last failing call.
 *   - "device" pointers are HIP device memory on the GPU that is current
 *     when gasloc_init runs; "host" pointers are ordinary CPU memory.
 *   - All device work is enqueued on the stream given to gasloc_init.  Only
 *     gasloc_consensus_error, gasloc_consensus_error_cols,
 *     gasloc_pseudo_gradient_sq and gasloc_destroy wait for the stream;
 *     kernel faults surface at the next blocking call.  A round that changes
 *     the CSR (or visit plan) stages it in a ring of four pinned host
 *     buffers, so it may wait until the stream has passed the upload made
 *     four uploads earlier (with all work enqueued before that upload).
 *   - A context is not thread-safe; distinct contexts are independent.
 *   - After a device error every call on the context returns GASLOC_ESTATE.
 *   - The library reads one environment variable, a test hook:
 *     GASLOC_GOSSIP_KERNEL=phase|planned forces the round kernel (by default
 *     the kernel that keeps every worker's value in LDS runs for n <= 16, the
 *     host-planned slot-reusing kernel beyond); results are bit-identical
 *     either way.
 */
#ifndef GASLOC_H
#define GASLOC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GASLOC_OK = 0,
  GASLOC_EINVAL = 1,  /* bad argument; nothing was enqueued                    */
  GASLOC_ENOMEM = 2,  /* host or device allocation failed                      */
  GASLOC_EDEVICE = 3, /* a HIP call failed (message has hipGetErrorString)     */
  GASLOC_ESTATE = 4   /* context unusable after an earlier device error        */
} gasloc_status;

typedef enum {
  GASLOC_F32 = 0, /* parameters x, y stored as fp32                             */
  GASLOC_BF16 = 1 /* parameters stored as bfloat16, rounded to nearest-even on
                     every store; optimizer state and arithmetic stay fp32      */
} gasloc_dtype;

/* Communication graph of a round, W = I - alpha * Lambda (section 3.1).
 * Every neighbourhood contains the worker itself (section 3.1, Notation);
 * neighbourhoods are sets, and unless stated the weights are 1/|N_i|
 * (Algorithm 1's average over N_i).  Columns are ascending within a row.
 * Cost: every graph gives the same results at any n, but beyond 16 workers
 * the round keeps each column's live values in LDS, so graphs whose distinct
 * rows need many of them at once run well below the HBM rate: the static
 * exponential graph (28 to 54 live) at n = 32-64 ran at 31-54% of peak
 * bandwidth, the sparse 1-Peer, 2-Peer, ring and random 3-regular graphs at
 * 63-77% (the low end where the buffers' physical placement is unfavourable:
 * the same round on other allocations runs at the high end).  Rows that are all the same (the complete graph, DiLoCo) share one
 * running sum instead: 63-77% of peak in fp32, 40-75% in bf16.  Use the
 * exponential graph beyond 16 workers for checks, not for speed. */
typedef enum {
  GASLOC_TOPO_EXPLICIT = 0,       /* the caller passes W to every round            */
  GASLOC_TOPO_RING = 1,           /* static cycle {i-1, i, i+1} (Tables 1-3 "ring")  */
  GASLOC_TOPO_COMPLETE = 2,       /* W = 11^T/n, i.e. Lambda = pi: DiLoCo (sec. 3.1)*/
  GASLOC_TOPO_EXPONENTIAL = 3,    /* static, directed: {i} u {i + 2^k mod n, 2^k < n}
                                     (exponential graph cited in section 3.2)      */
  GASLOC_TOPO_ONE_PEER_EXP = 4,   /* round t: {i, i + 2^(t mod tau) mod n},
                                     tau = ceil(log2 n), weights 1/2 (section 3.2) */
  GASLOC_TOPO_ONE_PEER = 5,       /* randomized 1-Peer (section 3.2, App. B.1): a
                                     fresh uniform permutation s per round, pairs
                                     (s[2k], s[2k+1]) mix 1/2-1/2; odd n leaves the
                                     last worker alone (W_ii = 1)                   */
  GASLOC_TOPO_TWO_PEER = 6,       /* randomized 2-Peer (section 3.2, App. B.1): s read
                                     as a cycle, each worker with both cyclic
                                     neighbours, weights 1/3                         */
  GASLOC_TOPO_RANDOM_REGULAR = 7  /* a fresh random `degree`-regular simple graph per
                                     round (pairing model with rejection), Metropolis
                                     weights 1/(1 + max(d_i, d_j))                   */
} gasloc_topology_kind;

/* Random graphs draw from SplitMix64 (Steele, Lea & Flood 2014) seeded per
 * round with mix(seed ^ mix(t)), mix = the SplitMix64 finalizer; bounded
 * draws reject values below 2^64 mod k; permutations are Fisher-Yates from
 * the identity.  The graph of round t is a pure function of (kind, n,
 * degree, seed, t): every worker agrees on it (App. B.1). */
typedef struct {
  int32_t kind;   /* gasloc_topology_kind                                        */
  int32_t degree; /* GASLOC_TOPO_RANDOM_REGULAR only: 0 <= degree < n, n*degree even */
  uint64_t seed;
  /* Optional (NULL = complete graph): host uint8 [n*n] row-major, symmetric,
   * 1 where an exchange is possible.  Restricts the ONE_PEER / TWO_PEER
   * selections to these edges (App. B.1); the weights are then
   * Metropolis-Hastings, which equal 1/2 and 1/3 when nothing is removed.
   * gasloc_init copies it. */
  const uint8_t *admissible;
} gasloc_topology;

/* How a round combines the workers' local iterates (the CSR W as below):
 *   EQ          z_i = x_i - eta (delta_i + mu u_i) with delta_i = x_i - y_i,
 *               x_i <- sum_j W_ij z_j + gamma (z_i - zp_i)    (Eq. 1 and Eq. 2,
 *               Nesterov outer step of section 4): the default
 *   ALG1        x_i <- OuterOpt(x_i, sum_j W_ij (x_i - y_j))      (Algorithm 1)
 *   DADAM       x_i <- sum_j W_ij x_j + (y_i - x_i)               (App. C)
 *   LOCAL_DADAM x_i <- OuterOpt(y_i, sum_j W_ij (x_i - x_j))      (App. C)
 * OuterOpt(b, d): u <- mu u + d; b - eta (d + mu u) (Nesterov) or b - eta u.
 * Only EQ uses gamma; DADAM uses neither eta nor mu nor u. */
typedef enum {
  GASLOC_FORM_EQ = 0,
  GASLOC_FORM_ALG1 = 1,
  GASLOC_FORM_DADAM = 2,
  GASLOC_FORM_LOCAL_DADAM = 3
} gasloc_round_form;

typedef struct {
  float beta1, beta2;          /* AdamW betas, 0 <= beta < 1 (paper: 0.9, 0.95)  */
  float eps;                   /* AdamW epsilon > 0 (added to sqrt(v_hat))       */
  float weight_decay;          /* decoupled weight decay >= 0 (paper: 0.1)       */
  float outer_lr;              /* eta > 0                                         */
  float outer_momentum;        /* mu in [0, 1); 0 gives Eq. 1's plain outer step   */
  int32_t outer_nesterov;      /* 1: Nesterov (z = x - eta (delta + mu u)),
                                  0: heavy ball (z = x - eta u)                   */
  float consensus_momentum;    /* gamma in [0, 1) of Eq. 2; 0 disables zp; must be
                                  0 unless round_form is EQ                       */
  int32_t param_dtype;         /* gasloc_dtype of x and y                          */
  int32_t round_form;          /* gasloc_round_form                                */
} gasloc_hparams;

/* Caller-owned device buffers, row-major [n, ld] with row i at offset i*ld.
 * Alignment: every pointer 16-byte aligned and ld * sizeof(element) a
 * multiple of 16.  Columns p >= P are never read or written.
 *   x  : round anchors x_t^i (param dtype)
 *   y  : live local iterates x_{t,h}^i (param dtype); see "deferred reset"
 *   m,v: AdamW moments (fp32)
 *   u  : outer momentum (fp32); may be NULL iff outer_momentum == 0 or the
 *        form is DADAM
 *   zp : previous post-outer iterate x_{t-1} + eta g_{t-1} (fp32);
 *        may be NULL iff consensus_momentum == 0                              */
typedef struct {
  void *x, *y;
  float *m, *v, *u, *zp;
  int64_t ld;
} gasloc_buffers;

/* A mixing matrix in CSR form, host memory: row_ptr[n+1] (row_ptr[0] = 0,
 * non-decreasing, row_ptr[n] = nnz), col[nnz] strictly ascending within a
 * row and in [0, n), val[nnz] finite fp32.  Accepted if every row sums to 1
 * within 1e-6 (in fp64).  Row i holds the weights worker i gives to its
 * neighbours: x_i <- sum_k val[k] * z_{col[k]}. */
typedef struct {
  int32_t n, nnz;
  const int32_t *row_ptr, *col;
  const float *val;
} gasloc_csr;

typedef struct gasloc_ctx gasloc_ctx;

/* Create a context for n in [1, 64] workers of P in [1, 2^31) parameters.
 * Validates the arguments, allocates the context's own small device scratch
 * (one CSR buffer, reduction partials) and a pinned CSR staging ring, zeroes m, v,
 * u, zp and the step counters on `hip_stream` (a hipStream_t; NULL = the
 * null stream).  The caller then fills x (and may leave y uninitialised):
 * y is logically equal to x until the first local step (identical start,
 * x_{t,0} = x_t in Eq. 1).  The buffers must outlive the context.
 * Errors: EINVAL for n, P, ld, alignment, NULL buffers, hyperparameters out
 * of range, bad topology (EXPLICIT is allowed: pass W to every round);
 * ENOMEM when a host or device allocation runs out of memory; EDEVICE for
 * any other HIP failure. */
gasloc_status gasloc_init(int32_t n, int64_t P, const gasloc_topology *topology,
                          const gasloc_hparams *hparams, const gasloc_buffers *buffers,
                          void *hip_stream, gasloc_ctx **out);

/* One local AdamW step (App. B "Optimization": decoupled weight decay,
 * bias-corrected moments, eps added to sqrt(v_hat)) for every worker i with
 * active[i] != 0 (active: host uint8[n]; NULL = all workers).  grads: device
 * fp32 [n, grad_ld], rows of inactive workers are not read.  Per element:
 *   w = y (1 - lr wd); m = b1 m + (1-b1) g; v = b2 v + (1-b2) g^2;
 *   y = w - lr/(1-b1^k) * m / (sqrt(v)/sqrt(1-b2^k) + eps)
 * with k the worker's step count after this step.  Inactive workers keep
 * their state and step count (heterogeneous H_i, section 3.2).  lr >= 0 is
 * the caller's schedule value for this step.  Enqueues one kernel. */
gasloc_status gasloc_local_step(gasloc_ctx *ctx, const float *grads, int64_t grad_ld,
                                const uint8_t *active, float lr);

/* One gossip round t (Eq. 1 outer loop with Eq. 2): for every worker i and
 * column p,
 *   delta = x - y;  u = mu u + delta;  z = x - eta (delta + mu u)  (Nesterov)
 *   x_i  = sum_k W_ik z_k  [+ gamma (z_i - zp_i) after the first round];
 *   zp_i = z_i  (if gamma != 0)
 * then the consensus error of the new x is reduced in fp64 and kept on the
 * device for gasloc_consensus_error.  W: the caller's CSR (host memory), or
 * NULL to use the context's topology for round t (EINVAL if EXPLICIT).
 * Deferred reset: afterwards y is logically equal to x but is not written;
 * the next local step of a worker reads x.  A worker that took no local
 * step since the last round has delta = 0.  Enqueues two kernels and one
 * host-to-device copy of the CSR (at most 33 KB). */
gasloc_status gasloc_gossip_round(gasloc_ctx *ctx, const gasloc_csr *W, uint64_t t);

/* One local step immediately followed by the gossip round, in a single pass
 * over HBM: the same results as gasloc_local_step(grads, grad_ld, active, lr)
 * then gasloc_gossip_round(W, t), bit for bit, but the new local iterate of
 * the stepping workers feeds the pseudo-gradient from registers and is never
 * stored (the round resets it to the new x anyway, Eq. 1: x_{t+1,0} =
 * x_{t+1}).  Use it for the last local step of a round (Algorithm 1: the
 * inner loop ends with y_i = x_i^{(t,H_i)}).  Saves 8 bytes per fp32
 * replica-parameter (12 when H_i = 1).  Same argument rules as the two calls;
 * EINVAL for the DADAM and LOCAL_DADAM forms (use the two calls there).
 * Enqueues two kernels and one CSR copy. */
gasloc_status gasloc_local_step_gossip_round(gasloc_ctx *ctx, const float *grads, int64_t grad_ld,
                                             const uint8_t *active, float lr, const gasloc_csr *W,
                                             uint64_t t);

/* ||pi x||^2 = sum_p sum_i (x_ip - xbar_p)^2 over the stored x (fp64
 * result).  Uses the value fused into the last gossip round when it is
 * current, otherwise reduces x afresh.  Blocks until the stream reaches it. */
gasloc_status gasloc_consensus_error(gasloc_ctx *ctx, double *out);

/* sum_i ||x_i - y_i||^2 over the pseudo-gradients the last gossip round
 * consumed (Eq. 1: g_t^i = x_{t,H} - x_{t,0}; y_i = x_i for a worker
 * without local steps; with the fused call, y_i is the iterate after the
 * fused step).  Differences in fp32, squares and sums in fp64, reduced inside
 * the round kernel at no extra HBM traffic.  0 before the first round.
 * Blocks until the stream reaches it. */
gasloc_status gasloc_pseudo_gradient_sq(gasloc_ctx *ctx, double *out);

/* The consensus error restricted to columns [p_begin, p_end) (0 <= p_begin <=
 * p_end <= P): one GPU's share when columns are split across GPUs.  Always
 * reduces x afresh.  Blocks. */
gasloc_status gasloc_consensus_error_cols(gasloc_ctx *ctx, int64_t p_begin, int64_t p_end,
                                          double *out);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * consensus error of gasloc_consensus_error_cols without a context.  x:
 * device [n, ld] in param_dtype (gasloc_dtype), 16-byte aligned, ld *
 * sizeof(param) a multiple of 16; columns [p_begin, p_end), 0 <= p_begin <=
 * p_end <= ld, p_end < 2^31; out: device, one fp64, 8-byte aligned, written
 * on hip_stream (the call does not wait), which must belong to the GPU that is
 * current on the calling thread (x and out live there, and so does the
 * scratch the call uses).  Same per-column arithmetic as
 * gasloc_consensus_error_cols; on ranges of at least 8 * 16 * 256 steps of
 * 1024 fp32 (2048 bf16) columns per CU it groups the sums the same way too.
 * Scratch: a fixed 512 KiB + 128 B device array inside the library (one copy
 * per GPU, held until the process ends); the call allocates nothing and calls
 * no allocating routine.  Limit: at most 2^16 workgroups of 8 x 256 column
 * groups, i.e. 2^29 fp32 or 2^30 bf16 columns per call (EINVAL beyond; the
 * error is additive over columns, so split the range and add the results).
 * Nothing in the scratch has to start at zero (every partial is written
 * before it is read).  Calls on one GPU share its scratch: calls that overlap
 * in time on one GPU (different streams, or different host threads) race;
 * calls in order on one stream do not.  Errors: EINVAL (checked before any
 * device work), EDEVICE. */
gasloc_status gasloc_consensus_error_cols_noalloc(const void *x, int32_t param_dtype, int32_t n, int64_t ld,
                                                  int64_t p_begin, int64_t p_end, double *out,
                                                  void *hip_stream);

/* Network average xbar_p = (1/n) sum_i x_ip (Algorithm 1 output), summed in
 * fp64 in worker order and rounded to the param dtype, into out (device,
 * [P] of the param dtype, 16-byte aligned).  Enqueues one kernel. */
gasloc_status gasloc_replica_mean(gasloc_ctx *ctx, void *out);

/* The context topology's W for round t, written to host arrays row_ptr[n+1],
 * col[cap], val[cap]; *nnz receives the entry count.  Host only.  EINVAL if
 * the context topology is EXPLICIT or cap is too small. */
gasloc_status gasloc_topology_csr(gasloc_ctx *ctx, uint64_t t, int32_t *row_ptr, int32_t *col,
                                  float *val, int32_t cap, int32_t *nnz);

/* Host-only schedule generator, no context and no device: the same W as
 * gasloc_topology_csr for the given topology and n. */
gasloc_status gasloc_make_topology(const gasloc_topology *topology, int32_t n, uint64_t t,
                                   int32_t *row_ptr, int32_t *col, float *val, int32_t cap,
                                   int32_t *nnz);

/* Local learning rate of step `step` (0-based, clamped to [0, total_steps])
 * under the schedule of App. B "Optimization": a linear warmup over the first
 * floor(warmup_frac * total_steps) steps from start_frac * peak to peak, then
 * a half-cosine decay to final_frac * peak at total_steps.  The paper's
 * setting is warmup_frac = 0.1, start_frac = 0.01 (final_frac unstated; 0 is
 * the usual choice).  Evaluated in fp64, returned in fp32.  Host only. */
float gasloc_lr_schedule(float peak, int64_t step, int64_t total_steps, float warmup_frac,
                         float start_frac, float final_frac);

/* Skipped exchanges (section 3.2, "Fault tolerance"), host only: W with
 * every exchange {i, j} removed whose worker i or j is dead (alive[.] == 0)
 * or whose link failed (link_ok[i*n + j] == 0 or link_ok[j*n + i] == 0);
 * each worker keeps the weight it would have given the other (W_ii += W_ij),
 * so rows still sum to 1 and a symmetric W stays doubly stochastic.  alive:
 * uint8[n] or NULL (all alive); link_ok: uint8[n*n] or NULL (all up).  Output
 * arrays as for gasloc_make_topology. */
gasloc_status gasloc_skip_exchanges(const gasloc_csr *W, const uint8_t *alive, const uint8_t *link_ok,
                                    int32_t *row_ptr, int32_t *col, float *val, int32_t cap,
                                    int32_t *nnz);

/* Marks workers dead or alive on a context (alive: host uint8[n]; NULL = all
 * alive).  From the next call on, the exchanges of dead workers are skipped
 * in every round's W (generated or passed in), as gasloc_skip_exchanges
 * does, and dead workers take no local steps whatever `active` says. */
gasloc_status gasloc_set_alive(gasloc_ctx *ctx, const uint8_t *alive);

/* Host-only CSR check with the rules listed at gasloc_csr (n must match). */
gasloc_status gasloc_validate_csr(const gasloc_csr *W, int32_t n);

/* Checkpoint / resume of the host-side counters: per-worker AdamW step counts
 * k[n], per-worker "stepped since the last round" flags stepped[n] (host
 * arrays, may be NULL to skip), rounds completed.  Together with the [n, P]
 * buffers and the topology seed this is the whole state of a run. */
gasloc_status gasloc_get_counters(const gasloc_ctx *ctx, int64_t *k, uint8_t *stepped,
                                  int64_t *rounds_done);
gasloc_status gasloc_set_counters(gasloc_ctx *ctx, const int64_t *k, const uint8_t *stepped,
                                  int64_t rounds_done);

/* Message of the last failing call on ctx; with ctx == NULL, of the last
 * failing context-free call (or gasloc_init) on this thread. */
const char *gasloc_last_error(const gasloc_ctx *ctx);

/* How this library was built: "sources <16 hex digits>; <arch>; <flags>",
 * the hex digits being the start of a SHA-256 over the source files it was
 * compiled from (paper_2606_11081_amd/build.py, sources_sha), so that a
 * caller can tell whether a prebuilt library matches a source tree.  A
 * static string; never NULL. */
const char *gasloc_build_info(void);

/* Wait for the context's stream, free its scratch; the caller's buffers are
 * untouched.  NULL is ignored. */
void gasloc_destroy(gasloc_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* GASLOC_H */
