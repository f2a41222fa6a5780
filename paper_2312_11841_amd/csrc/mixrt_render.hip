// The hot path: the fused per-pixel render kernel of the MixRT path for
// gfx950, and its launcher.
//
// render_kernel is one persistent kernel in which each wave repeatedly takes
// a tile of 64 sample slots (64/K rays x K samples), runs ray setup, Eq. 2
// calibration, contraction and the hash encoding with one sample per lane,
// stages the fp16 MLP inputs in its own slice of LDS, runs the MLP on MFMA
// with register-resident weights, and composites each ray's samples.  Nothing
// is written to HBM except the RGBA result.
#include "mixrt_common.hpp"
#include "mixrt_launch.hpp"

namespace mixrt {

// Levels per batch of corner loads in the render kernel.
constexpr int kLevelGroup = 2;

// A tile's R = 64/K rays cover a block of pixels, RW x RH with RW >= 4 RH,
// when R is a power of two (8 rays: 8 x 1; 64 rays: 16 x 4), else one row
// segment.  With one sample per ray the block puts nearby pixels in one wave,
// so its gathers share more cache lines (K = 1: 10-16% faster than a row of
// 64); with 8 samples per ray a row of 8 measured best.  Tiles never cross a
// row or view boundary.
struct TileShape {
    int RW, RH, tiles_x, per_view, n_tiles;
};

__host__ __device__ inline TileShape tile_shape(int R, int views, int W, int H)
{
    TileShape t;
    t.RH = 1;
    if ((R & (R - 1)) == 0)
        while (t.RH * t.RH * 16 <= R) t.RH *= 2;
    t.RW = R / t.RH;
    t.tiles_x = (W + t.RW - 1) / t.RW;
    t.per_view = t.tiles_x * ((H + t.RH - 1) / t.RH);
    t.n_tiles = views * t.per_view;
    return t;
}

// G levels of one query: into its fp16 row of MLP inputs, or (the MLP
// removed) added in fp32 to the per-component sums acc[(l F + i) mod 4].
template <int F, bool TF16, int G, bool DENSE, bool SUM>
__device__ __forceinline__ void encode_levels(const GridParams &gp, int l0, float x0, float x1,
                                              float x2, _Float16 *row, float *acc)
{
    float f[G][F];
    hash_group<F, TF16, G, DENSE>(gp, l0, x0, x1, x2, f);
#pragma unroll
    for (int g = 0; g < G; ++g) {
        if (SUM) {
            // F = 4: feature i feeds component i; F = 2: level parity picks 0-1 or 2-3
#pragma unroll
            for (int i = 0; i < F; ++i) {
                const int comp = (F == 4) ? i : (((l0 + g) & 1) * 2 + i);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (q == comp) acc[q] += f[g][i];
            }
        } else {
#pragma unroll
            for (int i = 0; i < F; i += 2)
                *(h2 *)(row + (l0 + g) * F + i) = h2{(_Float16)f[g][i], (_Float16)f[g][i + 1]};
        }
    }
}

// Stand-in for the weights when the MLP is removed.
struct NoMlp {
    __device__ __forceinline__ void load(const _Float16 *, int) {}
};

template <int TEX, int F, bool TF16, int IN, int HID, int NHID>
__global__ __launch_bounds__(kBlock) void render_kernel(RayParams rp, GridParams gp,
                                                        const _Float16 *__restrict__ weights,
                                                        int view_sh, float4 *__restrict__ out)
{
    typedef typename TexOf<TEX>::type TK;
    constexpr int LD = IN + 8;  // padded row of MLP inputs (halves), 16-byte multiple
    __shared__ __attribute__((aligned(16))) _Float16 s_rows[kWavesPerBlock][kWave * LD];
    __shared__ float4 s_out[kWavesPerBlock][kWave];
    __shared__ int s_hit[kWavesPerBlock][kWave];

    const int lane = threadIdx.x & (kWave - 1);
    // wave-uniform, so that the tile, its view and its camera live in scalar
    // registers (a lane-dependent view index makes the compiler keep every
    // camera in registers and select among them)
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    _Float16 *rows = s_rows[wv];

    // NHID = 0: the MLP removed; the level features are summed per component
    constexpr bool SUM = NHID == 0;
    typename std::conditional<SUM, NoMlp, MlpWeights<IN, HID, NHID>>::type Wt;
    Wt.load(weights, lane);

    const int K = rp.K;
    const int R = kWave / K;                 // rays per tile
    const int spt = R * K;                   // sample slots used per tile
    const TileShape ts = tile_shape(R, rp.views, rp.W, rp.H);
    const int gw = xcd_logical_block(blockIdx.x, gridDim.x) * kWavesPerBlock + wv;
    const int total = gridDim.x * kWavesPerBlock;
    const int r_loc = lane / K;
    const int k = lane - r_loc * K;
    const int L = gp.L;
    const int n_dense = gp.n_dense;

    for (int tile = gw; tile < ts.n_tiles; tile += total) {
        // the tile's pixel block, and ray r of it at (r % RW, r / RW)
        const int view = tile / ts.per_view, rem = tile - view * ts.per_view;
        const int ty = rem / ts.tiles_x, tx = rem - ty * ts.tiles_x;
        const int i0 = tx * ts.RW, j0 = ty * ts.RH;
        const int ray_base = (view * rp.H + j0) * rp.W + i0;
        const CamK &cam = rp.cams[view];
        auto ray_of = [&](int r, bool &in) {
            const int dy = r / ts.RW, dx = r - dy * ts.RW;
            in = r < R && i0 + dx < rp.W && j0 + dy < rp.H;
            return ray_base + dy * rp.W + dx;
        };
        bool in_img;
        const int ray = ray_of(r_loc, in_img);
        const bool valid = lane < spt && in_img;
        float x0 = 0.0f, x1 = 0.0f, x2 = 0.0f;
        bool hit = false;
        Ray ry = {};
        if (valid) {
            const int dy = r_loc / ts.RW, dx = r_loc - dy * ts.RW;
            ry = camera_ray(cam, rp.W, rp.H, (uint32_t)(i0 + dx), (uint32_t)(j0 + dy));
            hit = sample_position<TK>(rp, ry, rp.g0[ray], k, x0, x1, x2);
        }
        // --- hash encoding, features to LDS as fp16: dense levels first (pair
        // loads), then hashed levels, kLevelGroup levels per batch of loads
        _Float16 *row = rows + lane * LD;
        float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if (hit) {
            int l = 0;
            for (; l + kLevelGroup <= n_dense; l += kLevelGroup)
                encode_levels<F, TF16, kLevelGroup, true, SUM>(gp, l, x0, x1, x2, row, acc);
            for (; l < n_dense; ++l)
                encode_levels<F, TF16, 1, true, SUM>(gp, l, x0, x1, x2, row, acc);
            for (; l + kLevelGroup <= L; l += kLevelGroup)
                encode_levels<F, TF16, kLevelGroup, false, SUM>(gp, l, x0, x1, x2, row, acc);
            for (; l < L; ++l)
                encode_levels<F, TF16, 1, false, SUM>(gp, l, x0, x1, x2, row, acc);
        } else if (!SUM) {
            for (int e = 0; e < L * F; e += 2)
                *(h2 *)(row + e) = h2{(_Float16)0.0f, (_Float16)0.0f};
        }
        if (!SUM && view_sh) {
            float Y[16];
            sh_basis<16>(ry.dx, ry.dy, ry.dz, Y);
#pragma unroll
            for (int e = 0; e < 16; e += 2) {
                h2 hv = {(_Float16)(valid ? Y[e] : 0.0f), (_Float16)(valid ? Y[e + 1] : 0.0f)};
                *(h2 *)(row + L * F + e) = hv;
            }
        }
        if constexpr (SUM) {
            float4 a = mlp_activate(f4{acc[0], acc[1], acc[2], acc[3]});
            if (!hit) a.x = 0.0f;   // no density on a missed ray
            s_out[wv][lane] = a;
            wave_lds_sync();
        } else {
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
        }
        // --- compositing, one lane per ray
        if (lane < R) {
            bool in_c;
            const int ray_c = ray_of(lane, in_c);
            if (in_c) {
                Composite cp;
                for (int kk = 0; kk < K; ++kk)
                    if (!cp.add(s_out[wv][lane * K + kk], rp.delta, rp.t_term)) break;
                out[ray_c] = cp.finish(cam.bg[0], cam.bg[1], cam.bg[2]);
            }
        }
        wave_lds_sync();
    }
}


// Built render kernels: (texture kind, F, fp16 table, MLP in, hidden, hidden
// layers); in = hidden = layers = 0 is the MLP removed (any input width).
#define MIXRT_RENDER_VARIANTS(X)                \
    X(kTexF32Ray, 2, false, 16, 32, 1)          \
    X(kTexF32Ray, 2, false, 32, 32, 1)          \
    X(kTexF16Ray, 2, true, 48, 64, 2)           \
    X(kTexF16Ray, 2, true, 32, 64, 2)           \
    X(kTexF16Ray, 4, true, 32, 64, 2)           \
    X(kTexF16Ray, 4, true, 16, 64, 2)           \
    X(kTexU8Vec3D2, 4, true, 32, 64, 2)         \
    X(kTexF16Vec3D2, 4, true, 32, 64, 2)        \
    X(kTexF32Vec3D1, 2, false, 16, 32, 1)       \
    X(kTexU8Ray, 2, false, 16, 32, 1)           \
    X(kTexNone, 2, false, 16, 32, 1)            \
    X(kTexNone, 2, true, 48, 64, 2)             \
    X(kTexNone, 4, true, 32, 64, 2)             \
    X(kTexNone, 4, true, 32, 16, 2)             \
    X(kTexNone, 4, true, 0, 0, 0)               \
    X(kTexNone, 2, false, 0, 0, 0)              \
    X(kTexF32Ray, 2, false, 0, 0, 0)            \
    X(kTexU8Vec3D2, 4, true, 0, 0, 0)

bool render_variant_supported(int tex, int F, bool tf16, int in, int hid, int nhid)
{
#define X(a, b, c, d, e, f)                                                     \
    if (tex == a && F == b && tf16 == c && nhid == f && (f == 0 || (in == d && hid == e))) \
        return true;
    MIXRT_RENDER_VARIANTS(X)
#undef X
    return false;
}

// Persistent blocks per CU for a frame, given the most that fit (`resident`).
// More waves hide more latency when the gathers of a wave hit the same cache
// lines: several samples per ray, spaced finer than the cells of at least
// half the levels, on levels whose table fits one XCD's L2.  When the gathers
// scatter instead (one or two samples per ray, widely spaced samples, or
// levels larger than the L2), 2 blocks per CU keep more of each wave's lines
// in the caches and run faster than the full occupancy.  The count changes
// only which wave renders which tile, never a result.
static int render_blocks_per_cu(const RenderLaunch &L, int resident)
{
    if (L.blocks_mode == 1) return resident;
    if (L.blocks_mode == 2) return resident < 2 ? resident : 2;
    const float spacing = 0.25f * L.rp.delta;   // in grid units inside the unit ball
    int shared = 0;   // levels whose cells are at least one sample spacing wide
    for (int l = 0; l < L.gp.L; ++l)
        if ((float)L.gp.N[l] * spacing <= 1.0f) ++shared;
    const int64_t level_bytes = ((int64_t)L.gp.T_mask + 1) * L.F * (L.tf16 ? 2 : 4);
    const bool coherent = L.rp.K >= 4 && 2 * shared >= L.gp.L && level_bytes <= L.l2_bytes;
    return coherent || resident < 2 ? resident : 2;
}

hipError_t launch_render(const RenderLaunch &L, hipStream_t stream)
{
    const int R = kWave / L.rp.K;
    const int64_t n_tiles = tile_shape(R, L.rp.views, L.rp.W, L.rp.H).n_tiles;
    const int64_t want = (n_tiles + kWavesPerBlock - 1) / kWavesPerBlock;
#define X(a, b, c, d, e, f)                                                                    \
    if (L.tex == a && L.F == b && L.tf16 == c && L.nhid == f &&                                \
        (f == 0 || (L.in == d && L.hid == e))) {                                               \
        auto fn = render_kernel<a, b, c, d, e, f>;                                             \
        static std::atomic<int> per_cu{0};                                                     \
        /* blocks resident on the whole device */                                              \
        int64_t blocks =                                                                       \
            (int64_t)render_blocks_per_cu(L, blocks_per_cu((const void *)fn, per_cu)) * L.cus; \
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

}  // namespace mixrt
