// Stage kernels of the MixRT path (the entry points that expose one stage's
// intermediates): they call the same device functions as render_kernel.
#include "mixrt_common.hpp"
#include "mixrt_launch.hpp"

namespace mixrt {

template <int TEX>
__global__ __launch_bounds__(kBlock) void ray_setup_kernel(RayParams rp, float *__restrict__ out_x,
                                                           int32_t *__restrict__ out_hit)
{
    typedef typename TexOf<TEX>::type TK;
    const int64_t idx = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t n = (int64_t)rp.rays * rp.K;
    if (idx >= n) return;
    const int ray = (int)(idx / rp.K);
    const int k = (int)(idx - (int64_t)ray * rp.K);
    const Ray ry = pixel_ray(rp, ray);
    float x0, x1, x2;
    const bool hit = sample_position<TK>(rp, ry, rp.g0[ray], k, x0, x1, x2);
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
        // the render kernel's arithmetic, one level at a time (the render
        // kernel's queries lie in [0, 1]^3; here a coordinate outside it is
        // clamped to the grid)
        LevelSetup st;
        float v[8][F], f[F];
        const bool dense = l < gp.n_dense;
        constexpr uint32_t eb = TableEntry<F, TF16>::kBytes;
        level_setup<eb, false>(gp, l, dense, x0, x1, x2, st);
        const void *base = level_base(gp, l, F, TF16);
        if (dense)
            level_fetch<F, TF16, true>(base, st, v);
        else
            level_fetch<F, TF16, false>(base, st, v);
        level_accumulate<F>(st, v, f);
        const int64_t sl = s * gp.L + l;
        if (out_corner)
            for (int a = 0; a < 3; ++a) out_corner[sl * 3 + a] = (int32_t)st.cf[a];
        if (out_idx)
            for (int b = 0; b < 8; ++b) out_idx[sl * 8 + b] = st.off[b] / eb;
        if (out_w)
            for (int b = 0; b < 8; ++b) out_w[sl * 8 + b] = corner_weight(st, b);
        if (out_feat)
            for (int i = 0; i < F; ++i) out_feat[s * gp.L * F + l * F + i] = f[i];
    }
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"   // M0 is clobbered on purpose
// One 16-byte chunk per lane straight from global memory into LDS
// (global_load_lds_dwordx4): lane l's chunk lands at lds + 16 l.  M0 is set
// in the same statement; nothing else in this kernel uses it.  The rows are
// read once, so the load is marked non-temporal (nt), as are the output
// stores below: with both, the stage runs about 5% faster than with the
// default cache policy (0.161 against 0.169 ms for 7.37M rows), the writes
// disturbing the read stream less.
__device__ __forceinline__ void lds_load16(const void *g, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off nt" ::"s"(
                     __builtin_amdgcn_readfirstlane(lds)),
                 "v"(g)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

// A 16-byte non-temporal vector store, issued as assembly like the loads
// above.
__device__ __forceinline__ void store16(void *g, f4 v)
{
    asm volatile("global_store_dwordx4 %0, %1, off nt" ::"v"(g), "v"(v) : "memory");
}

// Wait until at most N vector-memory operations (loads and stores) of this
// wave are outstanding; they complete in issue order.
template <int N>
__device__ __forceinline__ void wait_vm()
{
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// wait_vm<n> for a wave-uniform n in 0..N
template <int N>
__device__ __forceinline__ void wait_vm_upto(int n)
{
    if constexpr (N == 0) {
        wait_vm<0>();
    } else {
        if (n >= N)
            wait_vm<N>();
        else
            wait_vm_upto<N - 1>(n);
    }
}

// Persistent: weights are loaded once per wave, then 64-row tiles.  A tile's
// rows are one contiguous block of 64 * CH 16-byte chunks, copied to LDS in
// CH coalesced loads, DEPTH tiles ahead of the one being computed; its 64
// outputs are gathered in LDS and written with one coalesced 1 KiB store
// (lane l: row l), the same access pattern as the stream the stage is
// measured against.
//
// The loads and stores of the tile loop are issued as assembly, so that the
// compiler, which sees no memory operation of its own there, places no wait
// of its own: its form of the LDS loads waits for every outstanding vector
// operation before any LDS read, and before inline assembly it drains its
// pending stores; either would serialise the pipelining.  The waits are
// counted instead.  Every tile issues exactly CH loads (the chunks of rows
// past n are read from the last row, and their outputs never stored) and
// exactly kStores stores (the lanes of rows past n masked off; a tile always
// has a row below n).  After the loads of tile k come the stores of the
// min(k, DEPTH) tiles before it and the loads of the tiles after it that are
// already in flight, and that is the count to wait for.
constexpr int kStores = 1;

template <int IN, int HID, int NHID, int DEPTH>
__global__ __launch_bounds__(kBlock) void mlp_kernel(const _Float16 *__restrict__ weights,
                                                     int hid_w, const _Float16 *__restrict__ in,
                                                     int64_t n, float4 *__restrict__ out4)
{
    static_assert(IN % 8 == 0, "rows are moved in 16-byte chunks");
    static_assert(DEPTH >= 1 && DEPTH <= 2, "tiles in flight");
    constexpr int CH = IN / 8;   // 16-byte chunks per row; a tile is CH 1-KiB loads
    constexpr int NB = DEPTH + 1;
    static_assert(DEPTH * (CH + kStores) <= 63, "vmcnt range");
    // NB tile buffers per wave, rows of IN halves back to back
    __shared__ __attribute__((aligned(16))) _Float16 s_rows[kWavesPerBlock][NB][kWave * IN];
    __shared__ f4 s_res[kWavesPerBlock][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    MlpWeights<IN, HID, NHID> Wt;
    Wt.load(weights, lane, hid_w);
    const int64_t n_tiles = (n + kWave - 1) / kWave;
    const int64_t total = (int64_t)gridDim.x * kWavesPerBlock;
    const int64_t first = (int64_t)blockIdx.x * kWavesPerBlock + wv;
    if (first >= n_tiles) return;
    const int count = (int)((n_tiles - 1 - first) / total) + 1;   // tiles of this wave
    const int64_t last_chunk = n * CH - 1;
    const h8 *chunks = (const h8 *)in;
    const int c = lane & 15, g = lane >> 4;
    auto issue = [&](int k) {
        const int64_t base = (first + (int64_t)k * total) * kWave * CH;
        const uint32_t lds = (uint32_t)(uintptr_t)s_rows[wv][k % NB];
#pragma unroll
        for (int e = 0; e < CH; ++e) {
            const int64_t q = base + lane + kWave * e;
            lds_load16(chunks + (q < last_chunk ? q : last_chunk), lds + 1024u * (uint32_t)e);
        }
    };
    for (int k = 0; k < DEPTH && k < count; ++k) issue(k);
    for (int k = 0; k < count; ++k) {
        if (k + DEPTH < count) issue(k + DEPTH);
        const int ahead = count - 1 - k < DEPTH ? count - 1 - k : DEPTH;
        const int stored = k < DEPTH ? k : DEPTH;
        wait_vm_upto<DEPTH *(CH + kStores)>(ahead * CH + stored * kStores);
        const _Float16 *rows = s_rows[wv][k % NB];
        const int64_t base = (first + (int64_t)k * total) * kWave;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const f4 o = mlp_tile<IN, HID, NHID>(Wt, rows + nt * 16 * IN, IN, lane);
            if (g == 0) {
                const float4 a = mlp_activate(o);
                s_res[wv][nt * 16 + c] = f4{a.x, a.y, a.z, a.w};
            }
        }
        wave_lds_sync();
        if (base + lane < n) store16(out4 + base + lane, s_res[wv][lane]);
    }
    wait_vm<0>();
}

// The MLP removed: inputs summed per component (input i feeds output i mod 4).
__global__ __launch_bounds__(kBlock) void sum_head_kernel(const _Float16 *__restrict__ in, int width,
                                                          int64_t n, float4 *__restrict__ out4)
{
    const int64_t s = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (s >= n) return;
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int i = 0; i < width; ++i) acc[i & 3] += (float)in[s * width + i];
    out4[s] = mlp_activate(f4{acc[0], acc[1], acc[2], acc[3]});
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

#define MIXRT_MLP_VARIANTS(X) \
    X(32, 16, 2)              \
    X(16, 32, 1)              \
    X(32, 32, 1)              \
    X(48, 64, 2)              \
    X(32, 64, 2)              \
    X(16, 64, 2)

bool mlp_variant_supported(int in, int hid, int nhid)
{
    if (nhid == 0) return in >= 4 && in % 4 == 0;
#define X(d, e, f) \
    if (in == d && hid == e && nhid == f) return true;
    MIXRT_MLP_VARIANTS(X)
#undef X
    return false;
}

hipError_t launch_ray_setup(const RayParams &rp, int tex, float *out_x, int32_t *out_hit,
                            hipStream_t stream)
{
    const int64_t n = (int64_t)rp.rays * rp.K;
    if (n == 0) return hipSuccess;
    const dim3 grid((unsigned)((n + kBlock - 1) / kBlock));
#define T(ID)                                                                                  \
    case ID:                                                                                   \
        hipLaunchKernelGGL(ray_setup_kernel<ID>, grid, dim3(kBlock), 0, stream, rp, out_x, out_hit); \
        break;
    switch (tex) {
        T(kTexF32Ray) T(kTexF16Ray) T(kTexU8Ray) T(kTexF32Vec3D1) T(kTexF16Vec3D2) T(kTexU8Vec3D2)
        T(kTexNone) T(kTexF32Vec3) T(kTexF16Vec3) T(kTexU8Vec3)
    default: return hipErrorInvalidValue;
    }
#undef T
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

// Tiles each wave has in flight beyond the one it computes.  One tile ahead
// leaves room in LDS for 3 blocks per CU (2 at two ahead) and, with the
// non-temporal loads and stores, runs about 2.5% faster (0.157 against 0.161
// ms for 7.37M rows of 48).
constexpr int kMlpDepth = 1;

hipError_t launch_mlp(int in, int hid, int nhid, int hid_w, const _Float16 *weights,
                      const _Float16 *x, int64_t n, float4 *out4, int cus, hipStream_t stream)
{
    if (n == 0) return hipSuccess;
    if (nhid == 0) {
        hipLaunchKernelGGL(sum_head_kernel, dim3((unsigned)((n + kBlock - 1) / kBlock)),
                           dim3(kBlock), 0, stream, x, in, n, out4);
        return hipGetLastError();
    }
    const int64_t want = ((n + kWave - 1) / kWave + kWavesPerBlock - 1) / kWavesPerBlock;
#define X(d, e, f)                                                                           \
    if (in == d && hid == e && nhid == f) {                                                  \
        auto fn = mlp_kernel<d, e, f, kMlpDepth>;                                            \
        static std::atomic<int> per_cu{0};                                                   \
        const int64_t resident = (int64_t)blocks_per_cu((const void *)fn, per_cu) * cus;     \
        const int64_t blocks = want < resident ? want : resident;                            \
        hipLaunchKernelGGL(fn, dim3((unsigned)blocks), dim3(kBlock), 0, stream, weights, hid_w, \
                           x, n, out4);                                                      \
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
