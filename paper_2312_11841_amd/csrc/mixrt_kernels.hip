// HIP kernels of the MixRT per-pixel path for gfx950, and their launchers.
//
// render_kernel is the hot path: one persistent kernel in which each wave
// repeatedly takes a tile of 64 sample slots (64/K rays x K samples), runs
// ray setup, Eq. 2 calibration, contraction and the hash encoding with one
// sample per lane, stages the fp16 MLP inputs in its own slice of LDS, runs
// the MLP on MFMA with register-resident weights, and composites each ray's
// samples.  Nothing is written to HBM except the RGBA result.
#include "mixrt_device.hpp"
#include "mixrt_launch.hpp"

namespace mixrt {

constexpr int kBlock = 256;             // 4 waves
constexpr int kWavesPerBlock = kBlock / kWave;

// Block -> logical block so that each XCD (blocks are dealt round-robin to
// the 8 XCDs) works on a contiguous range of tiles and shares its L2.
__device__ __forceinline__ int xcd_logical_block(int b, int nb)
{
    if (nb % 8 != 0) return b;
    return (b & 7) * (nb >> 3) + (b >> 3);
}

__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Levels per batch of corner loads in the render kernel.
constexpr int kLevelGroup = 2;

// G levels of one query into its fp16 row of MLP inputs.
template <int F, bool TF16, int G, bool DENSE>
__device__ __forceinline__ void encode_levels(const GridParams &gp, int l0, float x0, float x1,
                                              float x2, _Float16 *row)
{
    float f[G][F];
    hash_group<F, TF16, G, DENSE>(gp, l0, x0, x1, x2, f);
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
        for (int i = 0; i < F; i += 2)
            *(h2 *)(row + (l0 + g) * F + i) = h2{(_Float16)f[g][i], (_Float16)f[g][i + 1]};
    }
}

template <bool XF16, int F, bool TF16, int IN, int HID, int NHID>
__global__ __launch_bounds__(kBlock) void render_kernel(RayParams rp, GridParams gp,
                                                        const _Float16 *__restrict__ weights,
                                                        int view_sh, float4 *__restrict__ out)
{
    typedef typename std::conditional<XF16, _Float16, float>::type XT;
    constexpr int LD = IN + 8;  // padded row of MLP inputs (halves), 16-byte multiple
    __shared__ __attribute__((aligned(16))) _Float16 s_rows[kWavesPerBlock][kWave * LD];
    __shared__ float4 s_out[kWavesPerBlock][kWave];
    __shared__ int s_hit[kWavesPerBlock][kWave];

    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x / kWave;
    _Float16 *rows = s_rows[wv];

    MlpWeights<IN, HID, NHID> Wt;
    Wt.load(weights, lane);

    const int K = rp.K;
    const int R = kWave / K;                 // rays per tile
    const int spt = R * K;                   // sample slots used per tile
    const int n_tiles = (rp.rays + R - 1) / R;
    const int gw = xcd_logical_block(blockIdx.x, gridDim.x) * kWavesPerBlock + wv;
    const int total = gridDim.x * kWavesPerBlock;
    const int r_loc = lane / K;
    const int k = lane - r_loc * K;
    const int L = gp.L;
    const int n_dense = gp.n_dense;
    const uint32_t hw = (uint32_t)rp.H * (uint32_t)rp.W;

    for (int tile = gw; tile < n_tiles; tile += total) {
        const int ray0 = tile * R;
        const int ray = ray0 + r_loc;
        const bool valid = lane < spt && ray < rp.rays;
        float x0 = 0.0f, x1 = 0.0f, x2 = 0.0f;
        bool hit = false;
        Ray ry = {};
        if (valid) {
            ry = pixel_ray(rp, ray);
            hit = sample_position<XT>(rp, ry, rp.g0[ray], k, x0, x1, x2);
        }
        // --- hash encoding, features to LDS as fp16: dense levels first (pair
        // loads), then hashed levels, kLevelGroup levels per batch of loads
        _Float16 *row = rows + lane * LD;
        if (hit) {
            int l = 0;
            for (; l + kLevelGroup <= n_dense; l += kLevelGroup)
                encode_levels<F, TF16, kLevelGroup, true>(gp, l, x0, x1, x2, row);
            for (; l < n_dense; ++l)
                encode_levels<F, TF16, 1, true>(gp, l, x0, x1, x2, row);
            for (; l + kLevelGroup <= L; l += kLevelGroup)
                encode_levels<F, TF16, kLevelGroup, false>(gp, l, x0, x1, x2, row);
            for (; l < L; ++l)
                encode_levels<F, TF16, 1, false>(gp, l, x0, x1, x2, row);
        } else {
            for (int e = 0; e < L * F; e += 2)
                *(h2 *)(row + e) = h2{(_Float16)0.0f, (_Float16)0.0f};
        }
        if (view_sh) {
            float Y[16];
            sh_basis<16>(ry.dx, ry.dy, ry.dz, Y);
#pragma unroll
            for (int e = 0; e < 16; e += 2) {
                h2 hv = {(_Float16)(valid ? Y[e] : 0.0f), (_Float16)(valid ? Y[e + 1] : 0.0f)};
                *(h2 *)(row + L * F + e) = hv;
            }
        }
        s_hit[wv][lane] = hit ? 1 : 0;
        wave_lds_sync();
        // --- MLP on MFMA, 16 samples per step
        const int c = lane & 15, g = lane >> 4;
        const int n_nt = (spt + 15) >> 4;
        for (int nt = 0; nt < n_nt; ++nt) {
            const f4 o = mlp_tile<IN, HID, NHID>(Wt, rows + nt * 16 * LD, LD, lane);
            if (g == 0) {
                const int s = nt * 16 + c;
                float4 a = mlp_activate(o);
                if (!s_hit[wv][s]) a.x = 0.0f;   // no density on a missed ray
                s_out[wv][s] = a;
            }
        }
        wave_lds_sync();
        // --- compositing, one lane per ray
        if (lane < R) {
            const int ray_c = ray0 + lane;
            if (ray_c < rp.rays) {
                Composite cp;
                for (int kk = 0; kk < K; ++kk)
                    if (!cp.add(s_out[wv][lane * K + kk], rp.delta, rp.t_term)) break;
                const CamK &cam = rp.cams[(uint32_t)ray_c / hw];
                out[ray_c] = cp.finish(cam.bg[0], cam.bg[1], cam.bg[2]);
            }
        }
        wave_lds_sync();
    }
}

// --------------------------------------------------------------------------
// Stage kernels (the same device functions, outputs exposed)
// --------------------------------------------------------------------------

template <bool XF16>
__global__ __launch_bounds__(kBlock) void ray_setup_kernel(RayParams rp, float *__restrict__ out_x,
                                                           int32_t *__restrict__ out_hit)
{
    typedef typename std::conditional<XF16, _Float16, float>::type XT;
    const int64_t idx = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t n = (int64_t)rp.rays * rp.K;
    if (idx >= n) return;
    const int ray = (int)(idx / rp.K);
    const int k = (int)(idx - (int64_t)ray * rp.K);
    const Ray ry = pixel_ray(rp, ray);
    float x0, x1, x2;
    const bool hit = sample_position<XT>(rp, ry, rp.g0[ray], k, x0, x1, x2);
    out_x[idx * 3 + 0] = x0;
    out_x[idx * 3 + 1] = x1;
    out_x[idx * 3 + 2] = x2;
    if (out_hit && k == 0) out_hit[ray] = hit ? 1 : 0;
}

template <int F, bool TF16>
__global__ __launch_bounds__(kBlock) void hash_encode_kernel(GridParams gp, const float *__restrict__ x,
                                                             int64_t n, int32_t *out_corner,
                                                             uint32_t *out_idx, float *out_w,
                                                             float *out_feat)
{
    const int64_t s = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (s >= n) return;
    const float x0 = x[3 * s], x1 = x[3 * s + 1], x2 = x[3 * s + 2];
    for (int l = 0; l < gp.L; ++l) {
        // the render kernel's arithmetic, one level at a time
        LevelSetup st;
        float v[8][F], f[F];
        const bool dense = l < gp.n_dense;
        level_setup(gp.N[l], dense, gp.T_mask, x0, x1, x2, st);
        const void *base = level_base(gp, l, F, TF16);
        if (dense)
            level_fetch<F, TF16, true>(base, st, v);
        else
            level_fetch<F, TF16, false>(base, st, v);
        level_accumulate<F>(st, v, f);
        const int64_t sl = s * gp.L + l;
        if (out_corner)
            for (int a = 0; a < 3; ++a) out_corner[sl * 3 + a] = st.c[a];
        if (out_idx)
            for (int b = 0; b < 8; ++b) out_idx[sl * 8 + b] = st.idx[b];
        if (out_w)
            for (int b = 0; b < 8; ++b) out_w[sl * 8 + b] = corner_weight(st, b);
        if (out_feat)
            for (int i = 0; i < F; ++i) out_feat[s * gp.L * F + l * F + i] = f[i];
    }
}

template <int IN, int HID, int NHID>
__global__ __launch_bounds__(kBlock) void mlp_kernel(const _Float16 *__restrict__ weights,
                                                     const _Float16 *__restrict__ in, int64_t n,
                                                     float4 *__restrict__ out4)
{
    constexpr int LD = IN + 8;
    __shared__ __attribute__((aligned(16))) _Float16 s_rows[kWavesPerBlock][kWave * LD];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x / kWave;
    _Float16 *rows = s_rows[wv];
    MlpWeights<IN, HID, NHID> Wt;
    Wt.load(weights, lane);
    const int64_t base = ((int64_t)blockIdx.x * kWavesPerBlock + wv) * kWave;
    // stage 64 rows (zeros past n)
    const int64_t r = base + lane;
    for (int e = 0; e < IN; ++e)
        rows[lane * LD + e] = r < n ? in[r * IN + e] : (_Float16)0.0f;
    wave_lds_sync();
    const int c = lane & 15, g = lane >> 4;
    for (int nt = 0; nt < 4; ++nt) {
        const f4 o = mlp_tile<IN, HID, NHID>(Wt, rows + nt * 16 * LD, LD, lane);
        const int64_t s = base + nt * 16 + c;
        if (g == 0 && s < n) out4[s] = mlp_activate(o);
    }
}

__global__ __launch_bounds__(kBlock) void composite_kernel(const float4 *__restrict__ srgb,
                                                           int64_t rays, int K, float delta,
                                                           float t_term, float bg0, float bg1,
                                                           float bg2, float4 *__restrict__ out)
{
    const int64_t r = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (r >= rays) return;
    Composite cp;
    for (int k = 0; k < K; ++k)
        if (!cp.add(srgb[r * K + k], delta, t_term)) break;
    out[r] = cp.finish(bg0, bg1, bg2);
}

// --------------------------------------------------------------------------
// Launchers
// --------------------------------------------------------------------------

#define MIXRT_RENDER_VARIANTS(X)      \
    X(false, 2, false, 16, 32, 1)     \
    X(false, 2, false, 32, 32, 1)     \
    X(true, 2, true, 48, 64, 2)       \
    X(true, 2, true, 32, 64, 2)       \
    X(true, 4, true, 32, 64, 2)       \
    X(true, 4, true, 16, 64, 2)

#define MIXRT_MLP_VARIANTS(X) \
    X(16, 32, 1)              \
    X(32, 32, 1)              \
    X(48, 64, 2)              \
    X(32, 64, 2)              \
    X(16, 64, 2)

static int occupancy_blocks(const void *fn, int cus)
{
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, 0) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    return per_cu * cus;
}

bool render_variant_supported(bool xf16, int F, bool tf16, int in, int hid, int nhid)
{
#define X(a, b, c, d, e, f) \
    if (xf16 == a && F == b && tf16 == c && in == d && hid == e && nhid == f) return true;
    MIXRT_RENDER_VARIANTS(X)
#undef X
    return false;
}

bool mlp_variant_supported(int in, int hid, int nhid)
{
#define X(d, e, f) \
    if (in == d && hid == e && nhid == f) return true;
    MIXRT_MLP_VARIANTS(X)
#undef X
    return false;
}

hipError_t launch_render(const RenderLaunch &L, hipStream_t stream)
{
    const int R = kWave / L.rp.K;
    const int64_t n_tiles = ((int64_t)L.rp.rays + R - 1) / R;
    const int64_t want = (n_tiles + kWavesPerBlock - 1) / kWavesPerBlock;
#define X(a, b, c, d, e, f)                                                                    \
    if (L.xf16 == a && L.F == b && L.tf16 == c && L.in == d && L.hid == e && L.nhid == f) {     \
        auto fn = render_kernel<a, b, c, d, e, f>;                                             \
        static int resident = 0; /* blocks resident on the whole device */                    \
        if (!resident) resident = occupancy_blocks((const void *)fn, L.cus);                   \
        int64_t blocks = resident;                                                             \
        if (want < blocks) blocks = want;                                                      \
        if (blocks > 8) blocks -= blocks % 8;                                                  \
        if (blocks < 1) blocks = 1;                                                            \
        hipLaunchKernelGGL(fn, dim3((unsigned)blocks), dim3(kBlock), 0, stream, L.rp, L.gp,    \
                           L.weights, L.view_sh, L.out);                                       \
        return hipGetLastError();                                                              \
    }
    MIXRT_RENDER_VARIANTS(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_ray_setup(const RayParams &rp, bool xf16, float *out_x, int32_t *out_hit,
                            hipStream_t stream)
{
    const int64_t n = (int64_t)rp.rays * rp.K;
    if (n == 0) return hipSuccess;
    const dim3 grid((unsigned)((n + kBlock - 1) / kBlock));
    if (xf16)
        hipLaunchKernelGGL(ray_setup_kernel<true>, grid, dim3(kBlock), 0, stream, rp, out_x, out_hit);
    else
        hipLaunchKernelGGL(ray_setup_kernel<false>, grid, dim3(kBlock), 0, stream, rp, out_x,
                           out_hit);
    return hipGetLastError();
}

hipError_t launch_hash_encode(const GridParams &gp, int F, bool tf16, const float *x, int64_t n,
                              int32_t *oc, uint32_t *oi, float *ow, float *of, hipStream_t stream)
{
    if (n == 0) return hipSuccess;
    const dim3 grid((unsigned)((n + kBlock - 1) / kBlock));
#define LAUNCH(FF, TT)                                                                         \
    hipLaunchKernelGGL((hash_encode_kernel<FF, TT>), grid, dim3(kBlock), 0, stream, gp, x, n, oc, \
                       oi, ow, of)
    if (F == 2 && tf16) LAUNCH(2, true);
    else if (F == 2) LAUNCH(2, false);
    else if (F == 4 && tf16) LAUNCH(4, true);
    else if (F == 4) LAUNCH(4, false);
    else return hipErrorInvalidValue;
#undef LAUNCH
    return hipGetLastError();
}

hipError_t launch_mlp(int in, int hid, int nhid, const _Float16 *weights, const _Float16 *x,
                      int64_t n, float4 *out4, hipStream_t stream)
{
    if (n == 0) return hipSuccess;
    const int64_t per_block = (int64_t)kWavesPerBlock * kWave;
    const dim3 grid((unsigned)((n + per_block - 1) / per_block));
#define X(d, e, f)                                                                           \
    if (in == d && hid == e && nhid == f) {                                                  \
        hipLaunchKernelGGL((mlp_kernel<d, e, f>), grid, dim3(kBlock), 0, stream, weights, x, n, \
                           out4);                                                            \
        return hipGetLastError();                                                            \
    }
    MIXRT_MLP_VARIANTS(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_composite(const float4 *srgb, int64_t rays, int K, float delta, float t_term,
                            const float *bg, float4 *out, hipStream_t stream)
{
    if (rays == 0) return hipSuccess;
    const dim3 grid((unsigned)((rays + kBlock - 1) / kBlock));
    hipLaunchKernelGGL(composite_kernel, grid, dim3(kBlock), 0, stream, srgb, rays, K, delta,
                       t_term, bg[0], bg[1], bg[2], out);
    return hipGetLastError();
}

}  // namespace mixrt
