/*
 * mixrt_microbench.h -- roofline microbenchmarks for gfx950 (libmixrt_microbench.so).
 *
 * Not part of the rendering path: these kernels measure the achievable rates
 * the rendering kernel is compared against.  Each call enqueues one kernel on
 * `stream` (a hipStream_t, NULL for the null stream) and returns 0 or a
 * hipError_t code; the caller times it with events on that stream.  All
 * pointers are caller-owned device memory.
 */
#ifndef MIXRT_MICROBENCH_H
#define MIXRT_MICROBENCH_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Gathers from `table` (table_bytes, a power-of-two multiple of width):
 * blocks x 256 threads, each doing iters iterations of loads_per_iter (1 or
 * 8) independent loads of width (4, 8 or 16) bytes.  pattern 0: every lane
 * loads its own random element (one cache line per lane); pattern 1: all
 * lanes of a wave load the same element.  sink: device uint32 [blocks*256]
 * (written, keeps the loads live). */
int mixrt_mb_gather(const void *table, uint64_t table_bytes, int width, int loads_per_iter,
                    int iters, int pattern, int blocks, uint32_t *sink, void *stream);

/* Streaming copy of `bytes` (a multiple of 16) from src to dst with a
 * grid-stride loop over blocks x 256 threads. */
int mixrt_mb_copy(const void *src, void *dst, uint64_t bytes, int blocks, void *stream);

/* Streaming read of `bytes` (a multiple of 16) from src with a grid-stride
 * loop over blocks x 256 threads, four 16-byte loads per thread in flight;
 * sink: device uint32 [blocks*256] (written, keeps the loads live). */
int mixrt_mb_read(const void *src, uint64_t bytes, int blocks, uint32_t *sink, void *stream);

/* iters x 8 independent fp16 16x16x32 MFMAs per wave; blocks x 256 threads;
 * out: device float [blocks*256]. */
int mixrt_mb_mfma(int iters, int blocks, float *out, void *stream);

/* Properties of HIP device `device` the measurements are quoted against:
 * peak shader clock (kHz), memory clock (kHz), compute units, L2 bytes, and
 * the architecture name (NUL-terminated, at most cap bytes written). */
int mixrt_mb_device_info(int device, int *clock_khz, int *mem_clock_khz, int *cus,
                         int *l2_bytes, char *arch, int cap);

#ifdef __cplusplus
}
#endif

#endif /* MIXRT_MICROBENCH_H */
