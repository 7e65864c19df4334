/*
 * gasloc_probe.h -- measurement support in libgasloc.so: a streaming kernel
 * that moves the same byte mix as a kernel of the round, so that a benchmark
 * can state what a plain streaming kernel reaches on the same GPU, in the same
 * process, for that mix.  Not part of the method; the round never calls it.
 *
 * The probe kernel treats `count` elements of every stream as one flat
 * vector: each thread reads 4 consecutive elements of every source stream,
 * adds them in fp32 and stores the sum to 4 consecutive elements of every
 * destination stream (bf16 streams rounded to nearest-even).  Workgroups of
 * `threads` threads take one tile of 4 * threads elements each, dispatched
 * in order, as the round's kernels do.  Accesses are 16 bytes per lane for
 * fp32 streams and 8 for bf16 ones, non-temporal.  Which workgroup size
 * streams fastest depends on the mix (on MI355X, 64-thread workgroups are
 * a few percent faster on some mixes and slower on others), so a caller
 * after the achievable rate times several and keeps the fastest.
 */
#ifndef GASLOC_PROBE_H
#define GASLOC_PROBE_H

#include <stdint.h>

#include "gasloc.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Stream counts of the supported mixes (fp32 reads, bf16 reads, fp32 writes,
 * bf16 writes), with the kernel whose bytes per element they match:
 *   (4, 0, 0, 0)  read only
 *   (0, 0, 3, 0)  write only
 *   (1, 0, 1, 0)  copy
 *   (4, 0, 3, 0)  local AdamW step, fp32 parameters: y, g, m, v -> y, m, v;
 *                 also the EQ round with gamma != 0: x, y, u, zp -> x, u, zp
 *   (3, 0, 2, 0)  EQ round with gamma = 0, fp32 parameters: x, y, u -> x, u
 *   (3, 1, 2, 1)  local AdamW step, bf16 parameters
 *   (2, 2, 2, 1)  EQ round with gamma != 0, bf16 parameters
 *   (7, 0, 5, 0)  last local step fused into the EQ round, fp32 parameters
 *   (6, 0, 4, 0)  the same with gamma = 0
 *   (5, 2, 4, 1)  the same as (7, 0, 5, 0) with bf16 parameters
 * src: host array of device pointers, the fp32 streams first, then the bf16
 * ones; dst likewise.  A destination may be the same buffer as a source of the
 * same type (an in-place update, as in the round); otherwise streams must not
 * overlap.  Every pointer 16-byte aligned, each stream `count` elements,
 * count in [1, 2^31).  threads: the workgroup size, 64, 128 or 256.  sink: device, at least 4 bytes; written only by a
 * read-only mix, and only where the sum of a thread's elements is a NaN whose
 * bits are 0x7fc0dead (so that the reads cannot be optimised away; finite
 * inputs never write it).
 * Enqueues one kernel on hip_stream (a hipStream_t; NULL = the null stream).
 * Errors: EINVAL for an unsupported mix, NULL or misaligned pointers, count
 * out of range, threads not 64, 128 or 256; EDEVICE if the launch fails.  The
 * message is given by gasloc_last_error(NULL). */
gasloc_status gasloc_stream_probe(int32_t reads_f32, int32_t reads_bf16, int32_t writes_f32,
                                  int32_t writes_bf16, const void *const *src, void *const *dst,
                                  int64_t count, int32_t threads, void *sink, void *hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* GASLOC_PROBE_H */
