/* Test-only C program: whole rounds through the C ABI on the GPU with no
 * Python or torch in the process.  Device buffers come from hipMalloc; a
 * few local steps and gossip rounds (time-varying 2-Peer graph, gamma != 0,
 * the fused last step in the last round) run on the default stream, and the
 * stored x, the consensus error and the pseudo-gradient statistic are
 * compared with the fp32 oracle (linked from oracle/gasloc_oracle.c) fed the
 * same inputs.  Prints "c_device_consumer: ok" and exits 0 when the state is
 * bit-identical and the reductions agree to 1e-9 relative. */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "gasloc.h"

/* the fp32 oracle (REAL = float) */
int orc_topology(int kind, int n, int degree, uint64_t seed, uint64_t t, int32_t *row_ptr, int32_t *col,
                 float *val, int cap);
int orc_local_step(int n, int64_t P, int64_t ld, int dtype, void *y, const float *g, int64_t gld, float *m,
                   float *v, const uint8_t *active, const int64_t *k, double lr, double beta1, double beta2,
                   double eps, double wd);
int orc_gossip_round(int n, int64_t P, int64_t ld, int dtype, void *x, void *y, float *u, float *zp, float *z,
                     const int32_t *row_ptr, const int32_t *col, const float *val, double mu, double eta,
                     int nesterov, double gamma, int64_t rounds_done);
double orc_consensus_error(int n, int64_t P, int64_t ld, int dtype, const void *x);
double orc_pseudo_gradient_sq(int n, int64_t P, int64_t ld, int dtype, const void *x, const void *y);

#define N 6
#define P 1003
#define LD 1004

static int check(gasloc_status st, gasloc_ctx *ctx, const char *what) {
  if (st != GASLOC_OK) {
    fprintf(stderr, "%s: status %d: %s\n", what, (int)st, gasloc_last_error(ctx));
    return 1;
  }
  return 0;
}

static int hip_ok(hipError_t e, const char *what) {
  if (e != hipSuccess) {
    fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return 0;
  }
  return 1;
}

static uint64_t lcg = 0x9E3779B97F4A7C15ull;
static float draw(void) {
  lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
  return (float)((double)(lcg >> 11) / 9007199254740992.0 - 0.5);
}

static int rel_close(double a, double b) { return fabs(a - b) <= 1e-9 * fabs(b) + 1e-300; }

int main(void) {
  const size_t cells = (size_t)N * LD, bytes = sizeof(float) * cells;
  float *x0 = calloc(cells, sizeof(float)), *g = calloc(cells, sizeof(float));
  float *xo = calloc(cells, sizeof(float)), *yo = calloc(cells, sizeof(float));
  float *mo = calloc(cells, sizeof(float)), *vo = calloc(cells, sizeof(float));
  float *uo = calloc(cells, sizeof(float)), *zpo = calloc(cells, sizeof(float)), *zo = calloc(cells, sizeof(float));
  float *xg = calloc(cells, sizeof(float));
  if (!x0 || !g || !xo || !yo || !mo || !vo || !uo || !zpo || !zo || !xg) return 2;
  for (int64_t p = 0; p < P; ++p) {
    const float v = 0.02f * draw();
    for (int i = 0; i < N; ++i) x0[(size_t)i * LD + (size_t)p] = v; /* identical start */
  }
  memcpy(xo, x0, bytes);
  memcpy(yo, x0, bytes);

  float *x, *y, *m, *v, *u, *zp, *gd;
  float **bufs[] = {&x, &y, &m, &v, &u, &zp, &gd};
  for (int k = 0; k < 7; ++k)
    if (!hip_ok(hipMalloc((void **)bufs[k], bytes), "hipMalloc")) return 2;
  if (!hip_ok(hipMemcpy(x, x0, bytes, hipMemcpyHostToDevice), "hipMemcpy")) return 2;

  const gasloc_topology topo = {GASLOC_TOPO_TWO_PEER, 0, 3, NULL};
  const gasloc_hparams hp = {0.9f, 0.95f, 1e-8f, 0.1f, 0.7f, 0.9f, 1, 0.1f, GASLOC_F32, GASLOC_FORM_EQ};
  const gasloc_buffers b = {x, y, m, v, u, zp, LD};
  gasloc_ctx *ctx = NULL;
  if (check(gasloc_init(N, P, &topo, &hp, &b, NULL, &ctx), NULL, "gasloc_init")) return 1;

  const float lr = 4e-3f;
  int64_t k[N] = {0};
  uint8_t all[N];
  memset(all, 1, sizeof all);
  int32_t rp[N + 1], col[N * N];
  float val[N * N];
  int failures = 0;
  for (uint64_t t = 0; t < 3; ++t) {
    for (int h = 0; h < 2; ++h) {
      for (size_t c = 0; c < cells; ++c) g[c] = draw();
      if (!hip_ok(hipMemcpy(gd, g, bytes, hipMemcpyHostToDevice), "hipMemcpy")) return 2;
      for (int i = 0; i < N; ++i) ++k[i];
      orc_local_step(N, P, LD, 0, yo, g, LD, mo, vo, all, k, (double)lr, (double)hp.beta1, (double)hp.beta2,
                     (double)hp.eps, (double)hp.weight_decay);
      const int fused = t == 2 && h == 1;
      if (fused) {
        if (check(gasloc_local_step_gossip_round(ctx, gd, LD, NULL, lr, NULL, t), ctx, "fused round")) return 1;
      } else if (check(gasloc_local_step(ctx, gd, LD, NULL, lr), ctx, "local step")) {
        return 1;
      }
    }
    const double pg_ref = orc_pseudo_gradient_sq(N, P, LD, 0, xo, yo);
    if (t < 2 && check(gasloc_gossip_round(ctx, NULL, t), ctx, "round")) return 1;
    const int nnz = orc_topology(6 /* 2-Peer */, N, 0, 3, t, rp, col, val, N * N);
    if (nnz < N) return 2;
    orc_gossip_round(N, P, LD, 0, xo, yo, uo, zpo, zo, rp, col, val, (double)hp.outer_momentum,
                     (double)hp.outer_lr, 1, (double)hp.consensus_momentum, (int64_t)t);
    double ce = 0.0, pg = 0.0;
    if (check(gasloc_consensus_error(ctx, &ce), ctx, "consensus error")) return 1;
    if (check(gasloc_pseudo_gradient_sq(ctx, &pg), ctx, "pseudo-gradient")) return 1;
    const double ce_ref = orc_consensus_error(N, P, LD, 0, xo);
    if (!rel_close(ce, ce_ref) || !rel_close(pg, pg_ref)) {
      fprintf(stderr, "round %d: ce %.17g vs %.17g, pg %.17g vs %.17g\n", (int)t, ce, ce_ref, pg, pg_ref);
      ++failures;
    }
  }
  if (!hip_ok(hipMemcpy(xg, x, bytes, hipMemcpyDeviceToHost), "hipMemcpy")) return 2;
  for (int i = 0; i < N; ++i)
    for (int64_t p = 0; p < P; ++p) {
      const size_t e = (size_t)i * LD + (size_t)p;
      if (memcmp(&xg[e], &xo[e], sizeof(float)) != 0) {
        if (failures < 10) fprintf(stderr, "x[%d][%lld]: %.9g vs %.9g\n", i, (long long)p, xg[e], xo[e]);
        ++failures;
      }
    }
  gasloc_destroy(ctx);
  for (int q = 0; q < 7; ++q) (void)hipFree(*bufs[q]);
  free(x0); free(g); free(xo); free(yo); free(mo); free(vo); free(uo); free(zpo); free(zo); free(xg);
  if (failures) {
    fprintf(stderr, "%d mismatches\n", failures);
    return 1;
  }
  printf("c_device_consumer: ok\n");
  return 0;
}
