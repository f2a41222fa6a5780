/*
 * mixrt.h -- C ABI of the MI355X (gfx950) MixRT per-pixel rendering library.
 *
 * The library renders pixels the way "MixRT: Mixed Neural Representations
 * For Real-Time NeRF Rendering" (arXiv 2312.11841) describes its fragment
 * stage (Sec. 5.1.2 and Fig. 2): for every pixel, take the coarse-mesh hit
 * from a G-buffer (Fig. 2 step 1), calibrate it with the view-dependent
 * displacement map (Sec. 4.3.2, Eq. 2), place K samples along the ray around
 * the calibrated point, contract them (Sec. 2.1), query each in the
 * multiresolution hash grid (Sec. 3.1, 4.3.3), decode density and colour with
 * the small MLP (Sec. 3.1), and alpha-composite the samples (Sec. 3.1, Eq. 1).
 *
 * Conventions for every entry point:
 *  - Return value: MIXRT_OK (0) or a negative mixrt_status.  No exception
 *    crosses the ABI and the library never aborts the process.  On failure a
 *    message is available from mixrt_last_error() (per context) and from
 *    mixrt_thread_error() (per thread, also for calls without a context).
 *  - Device pointers are caller-owned device memory: the library reads or
 *    writes them only inside the work it enqueues and never frees or retains
 *    them.  Pointers to descriptors and cameras are host memory, read during
 *    the call only.
 *  - Work is enqueued asynchronously on the context's HIP stream; inputs
 *    must stay valid and unmodified until that work completes (e.g. until
 *    mixrt_sync()).  The same inputs give bitwise identical outputs.
 *  - Arrays are dense, row-major, in the layouts stated per field.
 */
#ifndef MIXRT_H
#define MIXRT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum mixrt_status {
    MIXRT_OK = 0,
    MIXRT_EINVAL = -1,        /* null pointer, bad size or inconsistent shape */
    MIXRT_ENOMEM = -2,        /* device (or, building a mesh, host) allocation failed */
    MIXRT_EDEVICE = -3,       /* HIP runtime error (launch or device failure) */
    MIXRT_EUNSUPPORTED = -4   /* valid request outside what this build serves */
};

/* Element types of stored arrays. */
enum mixrt_dtype { MIXRT_F32 = 0, MIXRT_F16 = 1, MIXRT_U8 = 2 };

/* Displacement forms (Eq. 2). */
enum mixrt_disp_mode {
    /* The V channels at p_t are coefficients of the first V real spherical
     * harmonics of the view direction d (bands by degree, m = -l..l); their
     * weighted sum s is a signed length and p_cali = p + s d. */
    MIXRT_DISP_ALONG_RAY = 0,
    /* Eq. 2 as printed: channel a*nb + v (nb = (sh_degree+1)^2, a = x, y, z)
     * is the coefficient of harmonic v for axis a; S = (sum_v Y_v(d) m[a*nb+v])_a
     * and p_cali = p + m_s(p_t) S with the scale map m_s. */
    MIXRT_DISP_SH_VEC3 = 1,
    /* No displacement map: p_cali = p. */
    MIXRT_DISP_NONE = 2
};

/* Context creation flags. */
enum mixrt_flags {
    MIXRT_FLAG_SYNC_CHECK = 1u,  /* synchronise after each call and report
                                    device errors as MIXRT_EDEVICE */
    /* Persistent blocks of the render kernel per CU.  By default a frame runs
     * every block that fits when a wave's gathers share cache lines (at least
     * 4 samples per ray, spaced finer than the cells of half the levels, on
     * levels whose table fits one XCD's L2) and 2 blocks per CU otherwise.
     * These force one choice (setting both is MIXRT_EINVAL); the choice
     * changes speed only, never a result. */
    MIXRT_FLAG_BLOCKS_FULL = 2u,
    MIXRT_FLAG_BLOCKS_TWO = 4u
};

#define MIXRT_MAX_VIEWS 16
#define MIXRT_MAX_LEVELS 32
#define MIXRT_MAX_TEX_CHANNELS 16
#define MIXRT_MAX_SAMPLES 64
#define MIXRT_MAX_LAYERS 8

typedef struct mixrt_ctx mixrt_ctx;

typedef struct {
    int32_t device;      /* HIP device ordinal; must be a gfx950 device */
    void *hip_stream;    /* hipStream_t the context enqueues on (NULL: the
                            device's null stream); caller-owned */
    uint32_t flags;      /* mixrt_flags */
    int32_t tile_stripe; /* order in which the render kernel's waves take the
                            image's tiles (speed only, never a result): 0 the
                            library's choice (stripes about 48 pixels wide),
                            > 0 vertical stripes of that many tiles, each
                            stripe row by row (compact blocks of pixels per
                            XCD), < 0 plain row-major order */
    int32_t early_stop_chunk; /* how mixrt_render evaluates a ray's samples
                            (speed only, never a result): > 0 front to back in
                            rounds of that many samples per ray (rounded down
                            to a power of two, at most K), a ray stopping once
                            its transmittance is below t_term; the rays still
                            running are packed into each round, so a stopped
                            ray costs no further gathers or MFMA work.  < 0
                            all K samples of a ray at once (the tile path).
                            0 the library's choice: the tile path for K < 4, K
                            not a power of two, or coherent samples on levels
                            larger than one XCD's L2; otherwise rounds of 4, 2
                            or 1 as a ray's samples share the voxels of at
                            least half, a quarter or fewer of the levels */
    int32_t block_levels; /* how many of the finest hash levels gather each
                            x-neighbour pair of corners as one aligned 16-byte
                            block holding both entries (tables of 2 or 4 fp16
                            features only; speed only, never a result): > 0
                            that many (hashed levels only), < 0 none, 0 the
                            library's choice (2 features: the three finest,
                            five in rounds of one sample per ray, four when a
                            level's table exceeds one XCD's L2 (eight at K >=
                            8), among the hashed levels finer than a ray's
                            sample spacing; 4 features: every hashed level
                            when there are 8 or more in tables of 2^10 or
                            more entries, else none) */
} mixrt_create_info;

/* The coarse-mesh hit per pixel (Fig. 2 step 1): rasterisation output. */
typedef struct {
    int32_t views, W, H; /* views * H * W pixels, view-major, row 0 at top */
    const float *g0;     /* device [views][H][W][4]: (t, u, v, unused); t is
                            the hit distance along the unit ray direction, a
                            pixel with !(t > 0 && isfinite(t)) is a miss;
                            (u, v) is the texture coordinate p_t.  16-byte
                            aligned. */
    const float *g1;     /* device [views][H][W][4] normal, or NULL; not read
                            (Eq. 2 uses the view direction, not the normal) */
} mixrt_gbuffer;

/* One view's pinhole camera (Sec. 3.1: rays r = o + t d through pixels).
 * OpenGL axes: the camera looks down -z with +y up; fov is vertical; pixel
 * (i, j) is sampled through its centre (i + 0.5, j + 0.5). */
typedef struct {
    float c2w[12];       /* camera-to-world, row-major 3x4 [R | o] */
    float fov_y_deg;     /* in (0, 180) */
    float bg[3];         /* background colour blended with the transmittance
                            left after the last sample */
} mixrt_camera;

/* View-dependent displacement map (Sec. 4.3.2, Eq. 2). */
typedef struct {
    int32_t R;           /* texture is R x R texels, addressed with texel
                            centres at (i + 0.5) / R, clamp to edge, row from v */
    int32_t V;           /* ALONG_RAY: channels used, 1..16 (ignored otherwise) */
    int32_t dtype;       /* MIXRT_F32, MIXRT_F16 or MIXRT_U8 */
    int32_t mode;        /* mixrt_disp_mode */
    const void *data;    /* device [R][R][C]; 16-byte aligned; NULL for NONE */
    int32_t C;           /* stored channels per texel, >= channels used; 0
                            means exactly the channels used.  Texels of a
                            multiple of 16 bytes are read with vector loads */
    int32_t sh_degree;   /* SH_VEC3: degree 0..3, 3 (sh_degree+1)^2 channels */
    const void *scale;   /* SH_VEC3: device [R][R] scale map m_s of dtype */
    float q_scale[2];    /* MIXRT_U8: value = q_offset + q_scale * q, for */
    float q_offset[2];   /* [0] the coefficient map and [1] the scale map
                            (the maps are quantised to 8 bits, Sec. 4.3.2) */
} mixrt_disp_tex;

/* Multiresolution hash grid (Sec. 3.1, 4.3.3, 5.1.2).  Level l has
 * resolution N_l = floor(N_min * b^l + 1e-6) with b = (N_max/N_min)^(1/(L-1))
 * and vertices 0..N_l per axis over the unit cube.  A level with
 * (N_l + 1)^3 <= T indexes its vertices densely (x fastest); other levels use
 * the spatial hash (v0 * 1 ^ v1 * 2654435761 ^ v2 * 805459861) mod T. */
typedef struct {
    int32_t L;           /* levels, 1..32 */
    int32_t log2_T;      /* T = 2^log2_T entries per level, 4..26 */
    int32_t F;           /* features per entry: 2 or 4 */
    int32_t N_min, N_max;/* 1 <= N_min <= N_max <= 2^20 */
    int32_t dtype;       /* MIXRT_F32 or MIXRT_F16 */
    const void *data;    /* device [L][T][F]; 16-byte aligned */
} mixrt_hash_grid;

/* The small MLP (Sec. 3.1): input [h ; e] where h is the level-major
 * concatenation of the L*F interpolated features and e the 16 real spherical
 * harmonics of the view direction when view_sh_dim = 16.  Hidden layers use
 * ReLU and no biases; the 4 outputs are (sigma_raw, r, g, b) with
 * sigma = exp(sigma_raw), rgb = sigmoid. */
typedef struct {
    int32_t n_layers;    /* weight matrices, 2..MIXRT_MAX_LAYERS; 0 = the MLP
                            removed (the ablation of Tab. 3): input i is added
                            to output i mod 4, width[0] a multiple of 4,
                            view_sh_dim 0, data unused */
    int32_t width[MIXRT_MAX_LAYERS + 1]; /* width[0] = L*F + view_sh_dim,
                            hidden widths equal (8, 16, 32 or 64; 8 runs on
                            the 16-wide MFMA tile with zero padding, which
                            computes the 8-wide network exactly), last = 4 */
    int32_t view_sh_dim; /* 0 or 16 */
    const uint16_t *data;/* device fp16 weights, layer m row-major
                            [width[m]][width[m+1]], layers concatenated;
                            16-byte aligned */
} mixrt_mlp;

/* Sampling around the calibrated point and compositing (Eq. 1). */
typedef struct {
    int32_t K;           /* samples per ray, 1..64, at offsets
                            (k - (K-1)/2) * delta along d */
    float delta;         /* sample spacing and the delta of Eq. 1, >= 0 */
    float t_term;        /* stop compositing a ray once its transmittance
                            drops below t_term (0: never), in [0, 1) */
} mixrt_sampling;

/* ---- lifecycle ---------------------------------------------------------- */

/* Create a context bound to ci->device and ci->hip_stream.  Fails with
 * MIXRT_EUNSUPPORTED unless the device is gfx950. *out is NULL on failure.
 * Allocates and zeroes the context's 10 KiB of render work counters on
 * ci->device and waits for the device to finish that (MIXRT_ENOMEM if the
 * allocation fails); the caller's current device is kept.
 * Renders of one context must not run at the same time (they share the
 * counters): keep them on its stream. */
int mixrt_create(mixrt_ctx **out, const mixrt_create_info *ci);

/* Release the context (not the caller's buffers or stream).  NULL is a
 * no-op.  Waits for the work pending on the context's stream, then frees
 * its work counters. */
int mixrt_destroy(mixrt_ctx *ctx);

/* Wait for all work enqueued by the context; MIXRT_EDEVICE on a device
 * error. */
int mixrt_sync(mixrt_ctx *ctx);

/* ---- validation (pure host: makes no HIP call, usable without a GPU) ------ */

/* Check every descriptor of a render call; writes a NUL-terminated message
 * of at most cap bytes to msg (may be NULL) on failure.  cams points to
 * gbuf->views cameras.  Returns the status mixrt_render would return for
 * these descriptors before launching anything. */
int mixrt_validate(const mixrt_gbuffer *gbuf, const mixrt_camera *cams,
                   const mixrt_disp_tex *disp, const mixrt_hash_grid *grid,
                   const mixrt_mlp *mlp, const mixrt_sampling *smp,
                   char *msg, size_t cap);

/* The level resolutions N_l of a grid (pure host).  out_N: host int32[L]. */
int mixrt_level_resolutions(const mixrt_hash_grid *grid, int32_t *out_N);

/* ---- the hot path ----------------------------------------------------------- */

/* Render views * H * W pixels into out_rgba (device float [views][H][W][4]:
 * composited rgb plus alpha = 1 - final transmittance).  A miss pixel gets
 * (bg, 0).  Enqueued on the context's stream; no device memory is allocated
 * (the kernels' work counters are the context's). */
int mixrt_render(mixrt_ctx *ctx, const mixrt_gbuffer *gbuf, const mixrt_camera *cams,
                 const mixrt_disp_tex *disp, const mixrt_hash_grid *grid,
                 const mixrt_mlp *mlp, const mixrt_sampling *smp, float *out_rgba);

/* For callers that cannot allocate device memory or own a per-context
 * buffer: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Renders exactly what mixrt_render renders (same
 * arguments, same kernels, same frame bit for bit), but the kernels' work
 * counters are one fixed array of the library's own device memory
 * (MIXRT_NOALLOC_SCRATCH_BYTES = 10 KiB per device, held until the process
 * ends), set up and zeroed by the first mixrt_create on that device; the
 * call makes no hipMalloc, hipFree or other allocating call.  The array's
 * size does not depend on the frame, so no frame is too large for it.  Every
 * call on a device shares that device's array: calls that overlap on one
 * device (other streams, other contexts, other threads) race and may skip
 * or repeat tiles.  Each launch leaves the counters at zero for the next. */
#define MIXRT_NOALLOC_SCRATCH_BYTES 10240
int mixrt_render_noalloc(mixrt_ctx *ctx, const mixrt_gbuffer *gbuf, const mixrt_camera *cams,
                         const mixrt_disp_tex *disp, const mixrt_hash_grid *grid,
                         const mixrt_mlp *mlp, const mixrt_sampling *smp, float *out_rgba);

/* How mixrt_render launches a frame (none of it changes a result). */
typedef struct {
    int32_t blocks;      /* persistent grid, blocks of 256 threads */
    int32_t tile_stripe; /* tile-order stripe width in tiles (the image's tile
                            columns for row-major order) */
    int32_t chunk;       /* samples per ray per round (0: all K at once) */
    int32_t block_from;  /* first hash level whose x-neighbour corner pairs
                            are gathered as 16-byte blocks (L: none) */
    int32_t hash_batch;  /* hashed levels per batch of gathers (2 or 4) */
    int32_t claims;      /* 1: each wave claims the last units of its XCD's
                            pool from the work counters; 0: every unit in the
                            fixed order */
} mixrt_launch_plan;

/* The launch mixrt_render would make for these descriptors on this
 * context; nothing is enqueued.  plan: host, written on success. */
int mixrt_render_launch_shape(mixrt_ctx *ctx, const mixrt_gbuffer *gbuf,
                              const mixrt_camera *cams, const mixrt_disp_tex *disp,
                              const mixrt_hash_grid *grid, const mixrt_mlp *mlp,
                              const mixrt_sampling *smp, mixrt_launch_plan *plan);

/* ---- stage entry points (the same device code as mixrt_render) ------------ */

/* Profiling: in the phase-timer build of the library (the same sources
 * compiled with -DMIXRT_PHASE_TIMER, which renders the same frames), every
 * wave of mixrt_render adds the shader clocks it spends in each phase of a
 * tile to device counters.  Waits for the device, then writes out (host
 * uint64[8]): [0] setup (ray, G-buffer, Eq. 2, samples, contraction),
 * [1] hash encoding, [2] MLP (with the view encoding), [3] compositing and
 * store, summed over waves; [4] tiles; [5] waves; [6] samples run through
 * the hash encoding and MLP (a hit ray's samples, and with early_stop_chunk
 * only those of rays still running); [7] zero.  reset != 0
 * zeroes the counters after reading.  MIXRT_EUNSUPPORTED in other builds. */
int mixrt_debug_phase_cycles(mixrt_ctx *ctx, uint64_t *out, int reset);

/* Steps before the grid: ray, hit, Eq. 2 calibration, K samples, contraction
 * and normalisation to [0,1]^3.  out_x: device float [views*H*W][K][3] (the
 * exact fp32 positions mixrt_render feeds to the grid; zeros for a miss).
 * out_hit: device int32 [views*H*W] (1 hit, 0 miss) or NULL. */
int mixrt_debug_ray_setup(mixrt_ctx *ctx, const mixrt_gbuffer *gbuf, const mixrt_camera *cams,
                          const mixrt_disp_tex *disp, const mixrt_sampling *smp,
                          float *out_x, int32_t *out_hit);

/* Hash-grid queries of n positions x (device float [n][3] in [0,1]^3).
 * Outputs (device, each may be NULL): out_corner int32 [n][L][3] lower voxel
 * corner; out_idx uint32 [n][L][8] table index of corner beta with offset
 * (beta&1, beta>>1&1, beta>>2&1); out_w float [n][L][8] trilinear weights;
 * out_feat float [n][L*F] level-major features. */
int mixrt_debug_hash_encode(mixrt_ctx *ctx, const mixrt_hash_grid *grid, const float *x,
                            int64_t n, int32_t *out_corner, uint32_t *out_idx,
                            float *out_w, float *out_feat);

/* The MLP on n fp16 inputs (device [n][width[0]], 16-byte aligned); out4:
 * device float [n][4] = (sigma, r, g, b) after exp / sigmoid, 16-byte
 * aligned. */
int mixrt_debug_mlp(mixrt_ctx *ctx, const mixrt_mlp *mlp, const uint16_t *in_f16, int64_t n,
                    float *out4);

/* Compositing of rays * K samples (device float [rays][K][4] =
 * (sigma, r, g, b)) over the background bg (host float[3]) into out_rgba
 * (device float [rays][4]), with smp->delta and smp->t_term. */
int mixrt_debug_composite(mixrt_ctx *ctx, const float *srgb, int64_t rays,
                          const mixrt_sampling *smp, const float *bg, float *out_rgba);

/* ---- geometry: the coarse-mesh hit per pixel (Fig. 2 step 1) -------------- */

/* The G-buffer the rendering path reads (g0: hit distance t and texture
 * coordinate p_t) is the intersection of each pixel's ray with the low-poly
 * mesh (Sec. 4.3, Fig. 2 step 1), which the paper obtains by rasterising the
 * mesh.  These entry points compute it by ray casting on the GPU instead: a
 * mesh is uploaded once into a uniform grid of triangle lists, then each
 * pixel's ray walks the grid cells it crosses and keeps the closest triangle
 * hit (t > MIXRT_RAY_T_MIN).  Hits at equal t go to the lower triangle index. */

#define MIXRT_RAY_T_MIN 1e-4f

typedef struct mixrt_mesh mixrt_mesh;

typedef struct {
    int64_t n_vertices;      /* 3 .. 2^31-1 */
    int64_t n_faces;         /* 1 .. 2^31-1 */
    const float *positions;  /* host [n_vertices][3], finite */
    const int32_t *faces;    /* host [n_faces][3] vertex indices in [0, n_vertices);
                                the face normal is e1 x e2 with e1 = p1 - p0,
                                e2 = p2 - p0 */
    const float *uv;         /* host [n_vertices][2] texture coordinates, or NULL
                                (then the G-buffer's p_t is (0, 0)) */
    int32_t grid_res[3];     /* ray-casting grid: cells per axis (1..1024 each, at most 2^26 in all),
                                or all 0: chosen from the bounds so that the
                                grid has about cells_per_face * n_faces cells */
    float cells_per_face;    /* for grid_res = 0; 0 means 8 */
} mixrt_mesh_desc;

typedef struct {
    int32_t grid_res[3];     /* cells per axis */
    float lo[3], hi[3];      /* the grid's box (the mesh bounds, padded) */
    int64_t n_faces;
    int64_t n_refs;          /* triangle entries over all cell lists */
    int64_t device_bytes;    /* device memory the mesh holds */
} mixrt_mesh_info;

/* Pure host (makes no HIP call): validate desc and report the grid that
 * mixrt_mesh_create would build for it (resolution, bounds, entries, device
 * bytes).  msg (may be NULL) receives a NUL-terminated message of at most
 * cap bytes on failure.  info may be NULL to validate only. */
int mixrt_mesh_plan(const mixrt_mesh_desc *desc, mixrt_mesh_info *info, char *msg, size_t cap);

/* Build the grid on the host (deterministic: each cell lists every triangle
 * whose plane crosses the cell and whose bounding box overlaps it, both with
 * the cell padded by 1/500 of its size, in ascending triangle order; empty
 * cells hold their Chebyshev distance to the nearest listed cell, which lets
 * the walk leap across empty space) and upload it to ctx's device: triangle
 * records in cell order (v0, e1, e2 and the triangle index), cell records,
 * per-triangle texture coordinates, and the triangle records once more in
 * triangle order (for mixrt_rasterize).  The mesh owns this device memory; the copies are
 * synchronous, so desc's arrays may be released on return.  *out is NULL on
 * failure (MIXRT_EINVAL for a bad descriptor, MIXRT_ENOMEM if the host
 * arrays of the build or the device memory cannot be allocated,
 * MIXRT_EUNSUPPORTED if the lists would reach 2^31 entries). */
int mixrt_mesh_create(mixrt_ctx *ctx, const mixrt_mesh_desc *desc, mixrt_mesh **out);

/* Sizes of a created mesh (host only). */
int mixrt_mesh_get_info(const mixrt_mesh *mesh, mixrt_mesh_info *info);

/* Free the mesh's device memory.  NULL is a no-op.  Work that reads the
 * mesh must have completed (hipFree synchronises the device). */
int mixrt_mesh_destroy(mixrt_mesh *mesh);

/* Ray-cast views * H * W pixels (the cameras and pixel rays of
 * mixrt_render) against the mesh, writing the G-buffer mixrt_render reads:
 * out_g0 (device float [views][H][W][4], 16-byte aligned) = (t, u, v, 0),
 * with t the distance along the unit ray direction and (u, v) the
 * barycentric interpolation of the hit triangle's vertex uv; a miss gets
 * (-1, 0, 0, 0).  out_g1 (device float [views][H][W][4], or NULL) = the unit
 * face normal and, in the fourth component, the bits of the int32 triangle
 * index (-1 for a miss).  The mesh must have been created on ctx's device.
 * Enqueued on the context's stream; no device memory is allocated. */
int mixrt_raycast(mixrt_ctx *ctx, const mixrt_mesh *mesh, int32_t views, int32_t W, int32_t H,
                  const mixrt_camera *cams, float *out_g0, float *out_g1);

/* The same G-buffer as mixrt_raycast (same per-pixel rays, same fp32
 * ray-triangle test, same closest-hit rule), computed the way the paper
 * obtains it: by rasterising the mesh (Fig. 2 step 1) with compute kernels
 * into a visibility buffer of (t, triangle) keys kept by atomic minimum.
 * Faster than mixrt_raycast for whole frames.  The keys live in out_g0
 * until the last of the call's three launches overwrites them, so no
 * device memory is allocated.  Fewer than 2^26 pixels per view
 * (MIXRT_EUNSUPPORTED beyond); other arguments as for mixrt_raycast. */
int mixrt_rasterize(mixrt_ctx *ctx, const mixrt_mesh *mesh, int32_t views, int32_t W, int32_t H,
                    const mixrt_camera *cams, float *out_g0, float *out_g1);

/* ---- errors ------------------------------------------------------------------- */

/* Static description of a status code. */
const char *mixrt_status_string(int status);

/* Message of the context's last failed call ("" if none); owned by the
 * context, valid until its next call or destruction. */
const char *mixrt_last_error(const mixrt_ctx *ctx);

/* Message of the calling thread's last failed call ("" if none); owned by
 * the library, valid until that thread's next call. */
const char *mixrt_thread_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MIXRT_H */
