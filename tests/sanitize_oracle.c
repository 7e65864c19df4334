/* Test-only driver for the oracle under AddressSanitizer and
 * UndefinedBehaviorSanitizer (built by tests/test_sanitizers.py together with
 * oracle/gasloc_oracle.c, once per precision): a few rounds of every round
 * form on every generated graph at small sizes with a ragged row stride,
 * fp32 and (in the fp32 build) bf16 parameters, skipped exchanges and the
 * reductions.  Exits 0 when every call succeeds. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#ifdef ORACLE_FP64
typedef double real;
#else
typedef float real;
#endif

int orc_topology(int kind, int n, int degree, uint64_t seed, uint64_t t, int32_t *row_ptr, int32_t *col,
                 real *val, int cap);
int orc_skip_exchanges(int n, const int32_t *row_ptr, const int32_t *col, const real *val,
                       const unsigned char *alive, const unsigned char *link_ok, int32_t *out_row_ptr,
                       int32_t *out_col, real *out_val, int cap);
int orc_local_step(int n, int64_t P, int64_t ld, int dtype, void *y, const float *g, int64_t gld, real *m,
                   real *v, const uint8_t *active, const int64_t *k, double lr, double beta1, double beta2,
                   double eps, double wd);
int orc_gossip_round(int n, int64_t P, int64_t ld, int dtype, void *x, void *y, real *u, real *zp, real *z,
                     const int32_t *row_ptr, const int32_t *col, const real *val, double mu, double eta,
                     int nesterov, double gamma, int64_t rounds_done);
int orc_alg1_round(int n, int64_t P, int64_t ld, int dtype, void *x, void *y, real *u, const int32_t *row_ptr,
                   const int32_t *col, const real *val, double mu, double eta, int nesterov);
int orc_dadam_round(int n, int64_t P, int64_t ld, int dtype, void *x, void *y, real *z, const int32_t *row_ptr,
                    const int32_t *col, const real *val);
int orc_local_dadam_round(int n, int64_t P, int64_t ld, int dtype, void *x, void *y, real *u, real *z,
                          const int32_t *row_ptr, const int32_t *col, const real *val, double mu, double eta,
                          int nesterov);
double orc_consensus_error(int n, int64_t P, int64_t ld, int dtype, const void *x);
double orc_pseudo_gradient_sq(int n, int64_t P, int64_t ld, int dtype, const void *x, const void *y);
void orc_replica_mean(int n, int64_t P, int64_t ld, int dtype, const void *x, void *out);

static int failures = 0;

static void expect(int ok, const char *what, int n, int kind, int form) {
  if (!ok) {
    fprintf(stderr, "FAIL %s (n=%d kind=%d form=%d)\n", what, n, kind, form);
    ++failures;
  }
}

static uint64_t lcg = 88172645463325252ull;
static double uniform(void) {
  lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
  return (double)(lcg >> 11) / 9007199254740992.0;
}

int main(void) {
  const int ns[] = {1, 2, 5, 8, 17, 33};
#ifdef ORACLE_FP64
  const int dtypes[] = {0};
  const int ndt = 1;
#else
  const int dtypes[] = {0, 1};
  const int ndt = 2;
#endif
  for (size_t a = 0; a < sizeof ns / sizeof ns[0]; ++a) {
    const int n = ns[a];
    const int64_t P = 37, ld = 41; /* ragged: the stride exceeds the row */
    const size_t cells = (size_t)n * (size_t)ld;
    for (int di = 0; di < ndt; ++di) {
      const int dtype = dtypes[di];
      const size_t psize = dtype == 1 ? 2 : sizeof(real);
      for (int kind = 1; kind <= 7; ++kind) {
        if (kind == 7 && (n < 4 || (3 * n) % 2)) continue;
        for (int form = 0; form < 4; ++form) {
          void *x = calloc(cells, psize), *y = calloc(cells, psize);
          real *m = calloc(cells, sizeof(real)), *v = calloc(cells, sizeof(real));
          real *u = calloc(cells, sizeof(real)), *zp = calloc(cells, sizeof(real));
          real *z = calloc(cells, sizeof(real));
          float *g = malloc(sizeof(float) * cells);
          void *mean = calloc((size_t)P, psize);
          int32_t *rp = malloc(sizeof(int32_t) * (size_t)(n + 1)), *col = malloc(sizeof(int32_t) * (size_t)(n * n));
          real *val = malloc(sizeof(real) * (size_t)(n * n));
          int32_t *srp = malloc(sizeof(int32_t) * (size_t)(n + 1)), *scol = malloc(sizeof(int32_t) * (size_t)(n * n));
          real *sval = malloc(sizeof(real) * (size_t)(n * n));
          uint8_t *active = malloc((size_t)n);
          unsigned char *alive = malloc((size_t)n);
          int64_t *k = calloc((size_t)n, sizeof(int64_t));
          if (!x || !y || !m || !v || !u || !zp || !z || !g || !mean || !rp || !col || !val || !srp || !scol ||
              !sval || !active || !alive || !k) {
            fprintf(stderr, "allocation failed\n");
            return 2;
          }
          for (uint64_t t = 0; t < 3; ++t) {
            for (int h = 0; h < 2; ++h) {
              for (size_t c = 0; c < cells; ++c) g[c] = (float)(uniform() - 0.5);
              for (int i = 0; i < n; ++i) {
                active[i] = (uint8_t)(uniform() < 0.8);
                if (active[i]) ++k[i];
              }
              expect(orc_local_step(n, P, ld, dtype, y, g, ld, m, v, active, k, 4e-3, 0.9, 0.95, 1e-8, 0.1) == 0,
                     "local_step", n, kind, form);
            }
            const int nnz = orc_topology(kind, n, 3, 5, t, rp, col, val, n * n);
            expect(nnz >= n, "topology", n, kind, form);
            if (nnz < n) continue;
            for (int i = 0; i < n; ++i) alive[i] = (unsigned char)(uniform() < 0.75);
            const int snnz = orc_skip_exchanges(n, rp, col, val, alive, NULL, srp, scol, sval, n * n);
            expect(snnz >= n, "skip_exchanges", n, kind, form);
            if (snnz < n) continue;
            int rc;
            if (form == 0)
              rc = orc_gossip_round(n, P, ld, dtype, x, y, u, zp, z, srp, scol, sval, 0.9, 0.7, 1, 0.1,
                                    (int64_t)t);
            else if (form == 1)
              rc = orc_alg1_round(n, P, ld, dtype, x, y, u, srp, scol, sval, 0.9, 0.7, 1);
            else if (form == 2)
              rc = orc_dadam_round(n, P, ld, dtype, x, y, z, srp, scol, sval);
            else
              rc = orc_local_dadam_round(n, P, ld, dtype, x, y, u, z, srp, scol, sval, 0.9, 0.7, 0);
            expect(rc == 0, "round", n, kind, form);
            const double ce = orc_consensus_error(n, P, ld, dtype, x);
            const double pg = orc_pseudo_gradient_sq(n, P, ld, dtype, x, y);
            expect(ce >= 0.0 && pg >= 0.0, "reductions", n, kind, form);
            orc_replica_mean(n, P, ld, dtype, x, mean);
          }
          free(x); free(y); free(m); free(v); free(u); free(zp); free(z); free(g); free(mean);
          free(rp); free(col); free(val); free(srp); free(scol); free(sval); free(active); free(alive); free(k);
        }
      }
    }
  }
  if (failures) {
    fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  printf("sanitize_oracle: ok\n");
  return 0;
}
