/* A plain C99 consumer of include/gasloc.h, built and run by
 * tests/test_c_header.py against libgasloc.so with no GPU: it uses only the
 * host-side calls (schedules, CSR validation, skipped exchanges, LR
 * schedule, the streaming probe's argument checks) and prints one line per
 * check. */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "gasloc.h"
#include "gasloc_probe.h"

int main(void) {
  enum { N = 8, CAP = N * N };
  int32_t rp[N + 1], col[CAP], nnz = 0;
  float val[CAP];
  gasloc_topology topo;
  memset(&topo, 0, sizeof topo);
  topo.kind = GASLOC_TOPO_EXPONENTIAL;
  topo.seed = 3;
  if (gasloc_make_topology(&topo, N, 0, rp, col, val, CAP, &nnz) != GASLOC_OK) {
    printf("make_topology failed: %s\n", gasloc_last_error(NULL));
    return 1;
  }
  printf("exponential n=%d nnz=%d row0=", N, nnz);
  for (int32_t k = rp[0]; k < rp[1]; ++k) printf(" %d:%g", col[k], val[k]);
  printf("\n");

  gasloc_csr W = {N, nnz, rp, col, val};
  printf("validate=%d\n", (int)gasloc_validate_csr(&W, N));
  float bad_val[CAP];
  memcpy(bad_val, val, sizeof bad_val);
  bad_val[0] = 2.0f; /* row 0 no longer sums to 1 */
  gasloc_csr bad = {N, nnz, rp, col, bad_val};
  printf("validate_bad=%d\n", (int)gasloc_validate_csr(&bad, N));

  uint8_t alive[N];
  for (int i = 0; i < N; ++i) alive[i] = (uint8_t)(i != 5);
  int32_t orp[N + 1], ocol[CAP], onnz = 0;
  float oval[CAP];
  if (gasloc_skip_exchanges(&W, alive, NULL, orp, ocol, oval, CAP, &onnz) != GASLOC_OK) {
    printf("skip_exchanges failed: %s\n", gasloc_last_error(NULL));
    return 1;
  }
  printf("dead5 row5=");
  for (int32_t k = orp[5]; k < orp[6]; ++k) printf(" %d:%g", ocol[k], oval[k]);
  printf("\n");

  printf("lr=%.9g %.9g %.9g\n", gasloc_lr_schedule(1e-3f, 0, 100, 0.1f, 0.01f, 0.0f),
         gasloc_lr_schedule(1e-3f, 10, 100, 0.1f, 0.01f, 0.0f), gasloc_lr_schedule(1e-3f, 99, 100, 0.1f, 0.01f, 0.0f));

  /* rejected before any device work: a mix no kernel has, a zero count, a
     workgroup size the probe does not launch */
  printf("probe_mix=%d\n", (int)gasloc_stream_probe(1, 1, 1, 1, NULL, NULL, 1024, 256, NULL, NULL));
  printf("probe_count=%d\n", (int)gasloc_stream_probe(1, 0, 1, 0, NULL, NULL, 0, 256, NULL, NULL));
  printf("probe_threads=%d\n", (int)gasloc_stream_probe(1, 0, 1, 0, NULL, NULL, 1024, 96, NULL, NULL));
  return 0;
}
