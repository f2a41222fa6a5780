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

/* Gathers of controlled line sharing: blocks x 256 threads, each wave doing
 * iters iterations of 8 independent width-byte (4, 8 or 16) loads, each load
 * instruction touching exactly `lines` distinct 128-byte lines of `table`
 * (lines divides 64; 64/lines lanes per line, consecutive lanes when
 * adjacent != 0, else lane l on line l mod lines).  table_bytes: a
 * power-of-two multiple of 128 (a small table stays in the vector L1, a
 * larger one in L2).  sink: device uint32 [blocks*256] (written). */
int mixrt_mb_gather_lines(const void *table, uint64_t table_bytes, int width, int lines,
                          int adjacent, int iters, int blocks, uint32_t *sink, void *stream);

/* Streaming copy of `bytes` (a multiple of 16) from src to dst with a
 * grid-stride loop over blocks x 256 threads. */
int mixrt_mb_copy(const void *src, void *dst, uint64_t bytes, int blocks, void *stream);

/* Streaming read of `bytes` (a multiple of 16) from src with a grid-stride
 * loop over blocks x 256 threads, four 16-byte loads per thread in flight;
 * sink: device uint32 [blocks*256] (written, keeps the loads live). */
int mixrt_mb_read(const void *src, uint64_t bytes, int blocks, uint32_t *sink, void *stream);

/* Mixed read/write stream in the MLP stage's pattern: rows (a multiple of
 * 64) rows of in_bytes (32, 64 or 96) read from src in tiles of 64 rows
 * (coalesced 16-byte loads), and 16 bytes per row written to dst (the XOR of
 * the row's chunks that the lane loaded); blocks x 256 threads, a wave per
 * tile, non-temporal loads and stores.  src: device [rows][in_bytes],
 * dst: device [rows][16], both 16-byte aligned. */
int mixrt_mb_rowstream(const void *src, void *dst, int64_t rows, int in_bytes, int blocks,
                       void *stream);

/* iters x 8 independent fp16 16x16x32 MFMAs per wave; blocks x 256 threads;
 * out: device float [blocks*256]. */
int mixrt_mb_mfma(int iters, int blocks, float *out, void *stream);

/* Gather replay of one frame's hash-grid loads, the floor of the render
 * kernel's gather stream: blocks x 256 threads, the render kernel's work
 * distribution (per-XCD pools: each wave's first rounds in a fixed order,
 * the rest claimed from counters in `work`, or with work NULL every unit in
 * the fixed order, as the render does when its plan's claims is 0) and tile
 * order (tile_stripe as returned by mixrt_render_launch_shape), one sample
 * per lane as in the render kernel;
 * each lane reads its sample's position from x (device float
 * [views*H*W][K][3], the frame's mixrt_debug_ray_setup output; rays with
 * hit[ray] == 0 are skipped, hit: device int32 [views*H*W]), computes the
 * level's voxel and corner offsets like the render kernel and issues the
 * same loads of `entry_bytes`-byte entries (4, 8 or 16) from `table`
 * (device [L][2^log2_T] entries, 16-byte aligned) in the same batches,
 * keeping only an XOR of the loaded words (mode 0).  Mode 1 issues no loads
 * (address arithmetic alone).  chunk: 0 replays the tile path (a tile's
 * K samples of R = 64/K rays per step); > 0 (a power of two dividing 64, at
 * most K) replays the early-termination path with rounds of chunk samples
 * as it runs when every ray hits and none stops (runs of K/chunk tiles per
 * wave, lane s*chunk + j on sample c*chunk + j of the run's ray s in round
 * c).  block_from: hashed levels from this one on (4-byte entries only) are
 * gathered as the render kernel gathers them there, one aligned 16-byte
 * block per x-neighbour corner pair plus the x + 1 entries of voxels that
 * straddle two blocks, one level per batch (as returned by
 * mixrt_render_launch_shape; L: none); hash_batch: hashed levels per batch
 * of the other gathers, 2 or 4 (4 only for entries of 8 or more bytes, as
 * the render kernel batches them).  N: host int32 [L], the level
 * resolutions (non-decreasing).  work: NULL or device uint32
 * [MIXRT_MB_WORK_WORDS], zero before the call and left at zero by it (one
 * buffer per stream: calls that overlap must not share it).  sink: device
 * uint32 [blocks*256] (written); with mode 0 the XOR over all of it is the
 * XOR of the 8 corner entries of every level of every hit sample. */
#define MIXRT_MB_WORK_WORDS 2560
int mixrt_mb_gather_replay(const float *x, const int32_t *hit, int32_t views, int32_t W,
                           int32_t H, int32_t K, const void *table, int32_t L, int32_t log2_T,
                           int32_t entry_bytes, const int32_t *N, int32_t tile_stripe,
                           int32_t chunk, int32_t block_from, int32_t hash_batch,
                           int32_t mode, int32_t blocks, uint32_t *work, uint32_t *sink,
                           void *stream);

/* Properties of HIP device `device` the measurements are quoted against:
 * peak shader clock (kHz), memory clock (kHz), compute units, L2 bytes, and
 * the architecture name (NUL-terminated, at most cap bytes written). */
int mixrt_mb_device_info(int device, int *clock_khz, int *mem_clock_khz, int *cus,
                         int *l2_bytes, char *arch, int cap);

#ifdef __cplusplus
}
#endif

#endif /* MIXRT_MICROBENCH_H */
