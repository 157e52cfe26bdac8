/*
 * Measurement probe of the benchmark (libtasq_probe.so), separate from the
 * TASQ library: it runs no part of the method and only measures the int8
 * matrix-instruction rate the GPU sustains with no memory traffic, the
 * compute ceiling that the benchmark reports beside the datasheet peak.
 */
#ifndef TASQ_PROBE_H
#define TASQ_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Launches `blocks` workgroups of 256 threads on `stream` (a hipStream_t,
 * NULL for the default stream); every wave issues iters rounds of
 * tasq_probe_mfma_chains() independent v_mfma_i32_32x32x32_i8 on register
 * operands (2 * 32 * 32 * 32 int8 ops each), then writes one int32 per
 * thread to sink (device memory owned by the caller, blocks * 256 int32).
 * Asynchronous; the caller times it with events on the same stream.
 * Returns 0, or -1 when blocks < 1, iters < 1, sink is NULL or the launch
 * fails.
 */
int tasq_probe_mfma_peak(int blocks, int iters, int32_t *sink, void *stream);

/* Independent matrix instructions per wave and iteration (8). */
int tasq_probe_mfma_chains(void);

#ifdef __cplusplus
}
#endif

#endif /* TASQ_PROBE_H */
