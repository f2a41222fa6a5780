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

// Profiling builds of this same source, selected with -D at compile time
// (the default build defines none of them; they exist to attribute the fused
// kernel's time to its stages, the way the paper's Tab. 3 removes stages):
//   MIXRT_SPLIT_NO_DISP  the displacement map is not read (p_cali = p);
//   MIXRT_SPLIT_NO_HASH  no table loads, every feature is zero (the sample
//                        positions are still computed and kept live);
//   MIXRT_SPLIT_NO_MLP   no MFMA: a sample's output is its first 4 features;
//   MIXRT_PHASE_TIMER    each wave adds the shader clocks it spends in each
//                        phase of a tile (setup, hash encoding, MLP,
//                        compositing) to phase_cycles, read back with
//                        mixrt_debug_phase_cycles.
// The split builds render wrong frames on purpose and are never the library
// the binding loads by default; the timer build renders the same frames.

namespace mixrt {

// Levels per batch of corner loads in the render kernel.
constexpr int kLevelGroup = 2;

#ifdef MIXRT_PHASE_TIMER
// [0..3] shader clocks summed over waves in setup, hash, MLP and compositing;
// [4] tiles; [5] waves; [6] samples run through the hash encoding and MLP
// (hit samples, and in the early-termination path only those of rays still
// running).
__device__ unsigned long long phase_cycles[8];
#define MIXRT_PHASE(i)                                          \
    do {                                                        \
        const uint64_t t_ = __builtin_readcyclecounter();       \
        ph[i] += t_ - t_last;                                   \
        t_last = t_;                                            \
    } while (0)
#else
#define MIXRT_PHASE(i) \
    do {               \
    } while (0)
#endif

// G levels of one query: into its fp16 row of MLP inputs, or (the MLP
// removed) added in fp32 to the per-component sums acc[(l F + i) mod 4].
template <int F, bool TF16, int G, bool DENSE, bool SUM, bool BLOCKS = false>
__device__ __forceinline__ void encode_levels(const GridParams &gp, int l0, float x0, float x1,
                                              float x2, _Float16 *row, float *acc)
{
    float f[G][F];
    hash_group<F, TF16, G, DENSE, BLOCKS>(gp, l0, x0, x1, x2, f);
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

// Every level of one query in order: dense levels, hashed levels with
// single-entry gathers (gp.hash_batch levels per batch, 4 only for entries
// of 8 or more bytes), then hashed levels from gp.block_from on with 16-byte
// block gathers: one level per batch for 4-byte entries (two levels' blocks
// in flight would cost a wave of occupancy), 2 for 8-byte ones (fp16 F = 4;
// batches of 4 raise these kernels' registers by about 40 and were 1-2%
// slower on 8 and 16 levels).
template <int F, bool TF16, bool SUM>
__device__ __forceinline__ void encode_query(const GridParams &gp, float x0, float x1, float x2,
                                             _Float16 *row, float *acc)
{
    const int L = gp.L, n_dense = gp.n_dense;
    int l = 0;
    for (; l + kLevelGroup <= n_dense; l += kLevelGroup)
        encode_levels<F, TF16, kLevelGroup, true, SUM>(gp, l, x0, x1, x2, row, acc);
    for (; l < n_dense; ++l)
        encode_levels<F, TF16, 1, true, SUM>(gp, l, x0, x1, x2, row, acc);
    const int lb = kBlockPairs<F, TF16> && gp.block_from < L ? max(gp.block_from, l) : L;
    if constexpr (kBlockPairs8<F, TF16>) {
        // 8-byte entries from gp.block_from on: 16-byte blocks of
        // x-neighbour pairs, 2 levels per batch
        if (gp.block_from < L) {
            // (l < gp.block_from is implied; spelled out, it keeps a dead
            // stack frame out of the texture-less kernel's build)
            for (; l < gp.block_from && l + kLevelGroup <= gp.block_from; l += kLevelGroup)
                encode_levels<F, TF16, kLevelGroup, false, SUM>(gp, l, x0, x1, x2, row, acc);
            for (; l < gp.block_from; ++l)
                encode_levels<F, TF16, 1, false, SUM>(gp, l, x0, x1, x2, row, acc);
            for (; l + kLevelGroup <= L; l += kLevelGroup)
                encode_levels<F, TF16, kLevelGroup, false, SUM, true>(gp, l, x0, x1, x2, row, acc);
            for (; l < L; ++l)
                encode_levels<F, TF16, 1, false, SUM, true>(gp, l, x0, x1, x2, row, acc);
            return;
        }
    }
    if constexpr (TableEntry<F, TF16>::kBytes >= 8) {
        if (gp.hash_batch >= 4)
            for (; l + 4 <= lb; l += 4)
                encode_levels<F, TF16, 4, false, SUM>(gp, l, x0, x1, x2, row, acc);
    }
    for (; l + kLevelGroup <= lb; l += kLevelGroup)
        encode_levels<F, TF16, kLevelGroup, false, SUM>(gp, l, x0, x1, x2, row, acc);
    for (; l < lb; ++l)
        encode_levels<F, TF16, 1, false, SUM>(gp, l, x0, x1, x2, row, acc);
    if constexpr (kBlockPairs<F, TF16>) {
        for (; l < L; ++l)
            encode_levels<F, TF16, 1, false, SUM, true>(gp, l, x0, x1, x2, row, acc);
    }
}

// Stand-in for the weights when the MLP is removed.
struct NoMlp {
    __device__ __forceinline__ void load(const _Float16 *, int, int) {}
};

// Kernels without an MLP or with hidden layers of 16 or fewer neurons always
// run at 2 blocks per CU (the light case of the blocks-per-CU rule: 2 waves
// per SIMD), so the compiler is told it may schedule for 2 waves instead of
// the most that fit.  Measured on Tab. 3's rows: 4 levels of 2^17 entries
// 12% faster, 8 and 16 levels within 1% either way.
#define MIXRT_LIGHT_WAVES(NHID, HID) \
    __attribute__((amdgpu_waves_per_eu(1, ((NHID) == 0 || (HID) <= 16) ? 2 : 8)))

template <int TEX, int F, bool TF16, int IN, int HID, int NHID>
__global__ __launch_bounds__(kBlock) MIXRT_LIGHT_WAVES(NHID, HID) void render_kernel(RayParams rp, GridParams gp,
                                                        const _Float16 *__restrict__ weights,
                                                        int view_sh, int hid_w, int stripe,
                                                        unsigned int *__restrict__ work,
                                                        float4 *__restrict__ out)
{
#ifdef MIXRT_SPLIT_NO_DISP
    typedef TexKind<float, kDispNone> TK;
#else
    typedef typename TexOf<TEX>::type TK;
#endif
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
    Wt.load(weights, lane, hid_w);

    const int K = rp.K;
    const int R = kWave / K;                 // rays per tile
    const int spt = R * K;                   // sample slots used per tile
    const TileShape ts = tile_shape(R, rp.views, rp.W, rp.H, stripe);
    const int r_loc = lane / K;
    const int k = lane - r_loc * K;
    const int L = gp.L;
    // tiles from the per-XCD pools (a counted tile's claim is in flight
    // while the tile before it is rendered)
    WorkPools pools(work, ts.n_tiles, lane);
#ifdef MIXRT_PHASE_TIMER
    uint64_t ph[4] = {0, 0, 0, 0}, n_tiles_done = 0, n_samples = 0;
    uint64_t t_last = __builtin_readcyclecounter();
#endif

    for (;;) {
        const int tile = pools.take(lane);
        if (tile < 0) break;
        // the tile's pixel block, and ray r of it at (r % RW, r / RW)
        const TilePos tp = tile_at(ts, tile);
        const int view = tp.view;
        const int i0 = tp.tx * ts.RW, j0 = tp.ty * ts.RH;
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
        MIXRT_PHASE(0);
#ifdef MIXRT_SPLIT_NO_HASH
        if (false) {
#else
        if (hit) {
#endif
            encode_query<F, TF16, SUM>(gp, x0, x1, x2, row, acc);
        } else if (!SUM) {
            for (int e = 0; e < L * F; e += 2)
                *(h2 *)(row + e) = h2{(_Float16)0.0f, (_Float16)0.0f};
        }
#ifdef MIXRT_SPLIT_NO_HASH
        // keep the sample positions (and so the ray setup) live
        row[0] = (_Float16)((x0 + x1 + x2) * 0.0f);
#endif
        MIXRT_PHASE(1);
        pools.prefetch(lane);
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
#ifdef MIXRT_SPLIT_NO_MLP
                const _Float16 *rr = rows + (nt * 16 + c) * LD;
                const f4 o = {(float)rr[0], (float)rr[1], (float)rr[2], (float)rr[3]};
#else
                const f4 o = mlp_tile<IN, HID, NHID>(Wt, rows + nt * 16 * LD, LD, lane);
#endif
                if (g == 0) {
                    const int s = nt * 16 + c;
                    float4 a = mlp_activate(o);
                    if (!s_hit[wv][s]) a.x = 0.0f;   // no density on a missed ray
                    s_out[wv][s] = a;
                }
            }
            wave_lds_sync();
        }
        MIXRT_PHASE(2);
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
        MIXRT_PHASE(3);
#ifdef MIXRT_PHASE_TIMER
        ++n_tiles_done;
        n_samples += __popcll(__ballot(hit));
#endif
    }
    pools.finish();
#ifdef MIXRT_PHASE_TIMER
    if (lane == 0) {
        for (int i = 0; i < 4; ++i) atomicAdd(&phase_cycles[i], (unsigned long long)ph[i]);
        atomicAdd(&phase_cycles[4], (unsigned long long)n_tiles_done);
        atomicAdd(&phase_cycles[5], 1ull);
        atomicAdd(&phase_cycles[6], (unsigned long long)n_samples);
    }
#endif
}


// ---------------------------------------------------------------------------
// Front to back with early termination that skips work (Eq. 1 stopped once
// the transmittance is below t_term).
//
// Each wave keeps up to NS = 64/C rays in flight, one per slot; slot s lives
// in the registers of lane s (its owner): the pixel, the ray's calibrated
// frame (P, d, t), its next sample index, and the compositing state.  A
// round evaluates the next C samples of every active slot (lane s C + j takes
// sample kn + j) with the same sample placement, hash encoding and MLP as
// render_kernel; each owner then composites its C samples in order, and a
// ray retires once its transmittance drops below t_term or its K samples are
// done.  Freed slots are refilled a whole tile at a time, with the tile's ray
// setup exactly as in render_kernel (64 lanes over R = 64/K rays); a missed
// ray gets the background at once and takes no slot.  So a ray that stops
// early issues no further gathers or MFMA work, and every pixel is
// composited from the same samples in the same order as render_kernel's.
// Needs C <= K and C dividing 64.
// ---------------------------------------------------------------------------
template <int TEX, int F, bool TF16, int IN, int HID, int NHID>
__global__ __launch_bounds__(kBlock) MIXRT_LIGHT_WAVES(NHID, HID) void render_queue_kernel(RayParams rp, GridParams gp,
                                                              const _Float16 *__restrict__ weights,
                                                              int view_sh, int hid_w, int stripe,
                                                              int C, unsigned int *__restrict__ work,
                                                              float4 *__restrict__ out)
{
#ifdef MIXRT_SPLIT_NO_DISP
    typedef TexKind<float, kDispNone> TK;
#else
    typedef typename TexOf<TEX>::type TK;
#endif
    constexpr int LD = IN + 8;  // padded row of MLP inputs (halves), 16-byte multiple
    __shared__ __attribute__((aligned(16))) _Float16 s_rows[kWavesPerBlock][kWave * LD];
    __shared__ float4 s_out[kWavesPerBlock][kWave];
    // slot frames: (P, t) and (d, pixel bits); the slot a staged ray goes to;
    // each view's background
    __shared__ float4 s_fa[kWavesPerBlock][kWave], s_fb[kWavesPerBlock][kWave];
    __shared__ int s_slot_of[kWavesPerBlock][kWave];
    __shared__ float4 s_bg[kMaxViews];

    const int lane = threadIdx.x & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    _Float16 *rows = s_rows[wv];
    if (threadIdx.x == 0)
        for (int v = 0; v < rp.views; ++v)
            s_bg[v] = make_float4(rp.cams[v].bg[0], rp.cams[v].bg[1], rp.cams[v].bg[2], 0.0f);
    __syncthreads();

    constexpr bool SUM = NHID == 0;
    typename std::conditional<SUM, NoMlp, MlpWeights<IN, HID, NHID>>::type Wt;
    Wt.load(weights, lane, hid_w);

    const int K = rp.K;
    const int R = kWave / K;                 // rays per tile
    const int spt = R * K;
    const TileShape ts = tile_shape(R, rp.views, rp.W, rp.H, stripe);
    const int NS = kWave / C;               // ray slots
    const int L = gp.L;

    // slot state of the owner lanes s < NS
    int s_ray = -1, s_kn = 0, s_view = 0;
    Composite cp;
    // A wave holds the rays of about K/C tiles at once, so it takes its tiles
    // in runs of B = K/C consecutive ones (the units of the per-XCD pools):
    // the rays in flight in a wave are neighbours, and an XCD's rays in
    // flight stay one compact block of the image.  The claim of a wave's
    // next run is in flight while the current run is admitted.
    const int B = K / C > 1 ? K / C : 1;
    WorkPools pools(work, (ts.n_tiles + B - 1) / B, lane);
    int run = 0, in_run = B;   // the first admission takes a run
#ifdef MIXRT_PHASE_TIMER
    uint64_t ph[4] = {0, 0, 0, 0}, n_tiles_done = 0, n_samples = 0;
    uint64_t t_last = __builtin_readcyclecounter();
#endif

    for (;;) {
        // --- admission: whole tiles while their rays fit in the empty slots
        for (;;) {
            const bool empty = lane < NS && s_ray < 0;
            const uint64_t em = __ballot(empty);
            if (run >= 0 && (in_run == B || (int64_t)run * B + in_run >= ts.n_tiles)) {
                // the run is used up (the last one may be short): take the next
                run = pools.take(lane);
                in_run = 0;
            }
            if (run < 0 || __popcll(em) < R) break;
            const int tile = run * B + in_run++;
#ifdef MIXRT_PHASE_TIMER
            ++n_tiles_done;
#endif
            const TilePos tp = tile_at(ts, tile);
            const int view = tp.view;
            const int i0 = tp.tx * ts.RW, j0 = tp.ty * ts.RH;
            const CamK &cam = rp.cams[view];
            const int r_loc = lane / K, k = lane - r_loc * K;
            const int dy = r_loc / ts.RW, dx = r_loc - dy * ts.RW;
            const bool valid = lane < spt && i0 + dx < rp.W && j0 + dy < rp.H;
            const int ray = (view * rp.H + j0 + dy) * rp.W + i0 + dx;
            Ray ry = {};
            RayHit h = {0.0f, 0.0f, 0.0f, 0.0f};
            bool hit = false;
            if (valid) {
                ry = camera_ray(cam, rp.W, rp.H, (uint32_t)(i0 + dx), (uint32_t)(j0 + dy));
                hit = ray_hit<TK>(rp, ry, rp.g0[ray], k, h);
            }
            const bool head = valid && k == 0;
            if (head && !hit) {
                Composite none;
                out[ray] = none.finish(cam.bg[0], cam.bg[1], cam.bg[2]);
            }
            const uint64_t hm = __ballot(head && hit);
            const int n_hit = __popcll(hm);
            // the q-th empty slot takes the q-th hit ray of the tile
            const int q_empty = __builtin_amdgcn_mbcnt_hi(
                (uint32_t)(em >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)em, 0u));
            if (empty) s_slot_of[wv][q_empty] = lane;
            wave_lds_sync();
            if (head && hit) {
                const int q = __builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(hm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)hm, 0u));
                const int sl = s_slot_of[wv][q];
                s_fa[wv][sl] = make_float4(h.px, h.py, h.pz, h.t);
                s_fb[wv][sl] = make_float4(ry.dx, ry.dy, ry.dz, __int_as_float(ray));
            }
            wave_lds_sync();
            if (empty && q_empty < n_hit) {
                s_ray = __float_as_int(s_fb[wv][lane].w);
                s_kn = 0;
                s_view = view;
                cp = Composite();
            }
        }
        if (__ballot(lane < NS && s_ray >= 0) == 0) break;   // no tile left either
        MIXRT_PHASE(0);

        // --- a round: lane s C + j evaluates sample kn + j of slot s
        const int sl = lane / C, j = lane - sl * C;
        const int kk = __shfl(s_kn, sl) + j;
        const bool live = __shfl(s_ray, sl) >= 0 && kk < K;
#ifdef MIXRT_PHASE_TIMER
        n_samples += __popcll(__ballot(live));
#endif
        const float4 fa = s_fa[wv][sl], fb = s_fb[wv][sl];
        const RayHit h = {fa.x, fa.y, fa.z, fa.w};
        float x0 = 0.0f, x1 = 0.0f, x2 = 0.0f;
        if (live) sample_at(rp, h, fb.x, fb.y, fb.z, kk, x0, x1, x2);
        _Float16 *row = rows + lane * LD;
        float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#ifdef MIXRT_SPLIT_NO_HASH
        if (false) {
#else
        if (live) {
#endif
            encode_query<F, TF16, SUM>(gp, x0, x1, x2, row, acc);
        } else if (!SUM) {
            for (int e = 0; e < L * F; e += 2)
                *(h2 *)(row + e) = h2{(_Float16)0.0f, (_Float16)0.0f};
        }
#ifdef MIXRT_SPLIT_NO_HASH
        row[0] = (_Float16)((x0 + x1 + x2) * 0.0f);
#endif
        MIXRT_PHASE(1);
        pools.prefetch(lane);
        if (!SUM && view_sh) {
            float Y[16];
            sh_basis<16>(fb.x, fb.y, fb.z, Y);
#pragma unroll
            for (int e = 0; e < 16; e += 2) {
                h2 hv = {(_Float16)(live ? Y[e] : 0.0f), (_Float16)(live ? Y[e + 1] : 0.0f)};
                *(h2 *)(row + L * F + e) = hv;
            }
        }
        if constexpr (SUM) {
            float4 a = mlp_activate(f4{acc[0], acc[1], acc[2], acc[3]});
            if (!live) a.x = 0.0f;
            s_out[wv][lane] = a;
            wave_lds_sync();
        } else {
            wave_lds_sync();
            const int c = lane & 15, g = lane >> 4;
            for (int nt = 0; nt < kWave / 16; ++nt) {
#ifdef MIXRT_SPLIT_NO_MLP
                const _Float16 *rr = rows + (nt * 16 + c) * LD;
                const f4 o = {(float)rr[0], (float)rr[1], (float)rr[2], (float)rr[3]};
#else
                const f4 o = mlp_tile<IN, HID, NHID>(Wt, rows + nt * 16 * LD, LD, lane);
#endif
                if (g == 0) s_out[wv][nt * 16 + c] = mlp_activate(o);
            }
            wave_lds_sync();
        }
        MIXRT_PHASE(2);
        // --- compositing: each owner adds its slot's C samples in order
        if (lane < NS && s_ray >= 0) {
            bool going = true;
            for (int jj = 0; jj < C && going; ++jj) {
                if (s_kn + jj >= K) break;
                going = cp.add(s_out[wv][lane * C + jj], rp.delta, rp.t_term);
            }
            s_kn += C;
            if (!going || s_kn >= K) {
                const float4 bg = s_bg[s_view];
                out[s_ray] = cp.finish(bg.x, bg.y, bg.z);
                s_ray = -1;
            }
        }
        wave_lds_sync();
        MIXRT_PHASE(3);
    }
    pools.finish();
#ifdef MIXRT_PHASE_TIMER
    if (lane == 0) {
        for (int i = 0; i < 4; ++i) atomicAdd(&phase_cycles[i], (unsigned long long)ph[i]);
        atomicAdd(&phase_cycles[4], (unsigned long long)n_tiles_done);
        atomicAdd(&phase_cycles[5], 1ull);
        atomicAdd(&phase_cycles[6], (unsigned long long)n_samples);
    }
#endif
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
    X(kTexU8Vec3D2, 4, true, 0, 0, 0)           \
    X(kTexF32Vec3, 2, false, 16, 32, 1)         \
    X(kTexF16Vec3, 2, false, 16, 32, 1)         \
    X(kTexU8Vec3, 2, false, 16, 32, 1)          \
    X(kTexF32Vec3, 4, true, 32, 64, 2)          \
    X(kTexF16Vec3, 4, true, 32, 64, 2)          \
    X(kTexU8Vec3, 4, true, 32, 64, 2)

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
// More waves hide more latency, except where a wave's gathers touch so many
// lines that fewer waves keep more of each one's lines in the caches: rays
// whose K >= 4 samples lie apart on most levels (spaced coarser than the
// cells of half the levels), and kernels without an MLP or with one of
// hidden width 16 or less (Tab. 3's 2 x 8), whose waves do little besides
// gathering (their kernels are compiled for 2 waves per SIMD).  There 2
// blocks per CU run faster than the full occupancy.  Large tables (8 MiB
// levels) and one or two samples per ray also wanted 2 blocks per CU while
// every unit went in the fixed order; with each XCD's last units claimed from
// counters its working set stays compact and the full occupancy wins there
// (7-17%).  The count changes only which wave renders which tile, never a
// result.
static int levels_shared_by_samples(const RenderLaunch &L);

static int render_blocks_per_cu(const RenderLaunch &L, int resident)
{
    if (L.blocks_mode == 1) return resident;
    if (L.blocks_mode == 2) return resident < 2 ? resident : 2;
    const bool scattered = L.rp.K >= 4 && 2 * levels_shared_by_samples(L) < L.gp.L;
    const bool light = L.nhid == 0 || L.hid_w <= 16;
    return (scattered || light) && resident > 2 ? 2 : resident;
}

// Tile order for a frame (the stripe width of tile_at, in tiles).  Waves
// take tiles in order and the blocks are dealt to the 8 XCDs in contiguous
// runs, so the tiles one XCD renders at once are a run of the order; in
// stripes of about 48 pixels that run is a compact block of the image
// instead of a strip along rows, and neighbouring pixels' samples, which
// share voxel corners, meet in the same L2.  Measured on 16 workloads (K 1 to
// 32, 720p and the 8-view 1080p batch): 48-pixel stripes were 1-13% faster
// than row-major order everywhere and within 1.5% of each workload's best
// stripe on most of them (4.5% at worst).
static int render_stripe(const RenderLaunch &L, const TileShape &ts, int64_t blocks)
{
    (void)blocks;
    constexpr int kStripePixels = 48;
    if (L.tile_stripe < 0) return ts.tiles_x;
    int st = L.tile_stripe > 0 ? L.tile_stripe : (kStripePixels + ts.RW / 2) / ts.RW;
    if (st < 1) st = 1;
    return st < ts.tiles_x ? st : ts.tiles_x;
}

// Levels whose cells are at least one sample spacing wide (inside the unit
// ball the cube map divides lengths by 4): on these a ray's consecutive
// samples mostly share their voxel and its table lines.
static int levels_shared_by_samples(const RenderLaunch &L)
{
    const float spacing = 0.25f * L.rp.delta;   // in grid units inside the unit ball
    int shared = 0;
    for (int l = 0; l < L.gp.L; ++l)
        if ((float)L.gp.N[l] * spacing <= 1.0f) ++shared;
    return shared;
}

// Samples per ray per round of the early-termination path (0: the tile
// path).  A power of two dividing 64, at most K: the context's explicit
// request, or by default (measured at 720p and on the 8-view 1080p batch, K
// 2 to 32, spacings 0.01 to 0.25):
//  - K below 4 or not a power of two: the tile path (rounds would leave
//    lanes idle or gain nothing);
//  - a ray's samples share the voxels of at least half the levels: rounds
//    of 4 (3-30% faster than the tile path with no ray stopping, 16-66% on
//    opaque content), unless a level's table exceeds one XCD's L2 (the
//    batch: 5% slower, the tile path kept);
//  - at least a quarter: rounds of 2 (9% faster at spacing 0.05);
//  - fewer: rounds of 1, one sample of each of 64 neighbouring rays per
//    gather instruction, which share lines where a ray's own samples no
//    longer do (13-45% faster at spacing 0.25).
static int render_chunk(const RenderLaunch &L)
{
    const int K = L.rp.K;
    int want = L.chunk;
    if (want < 0) return 0;
    if (want == 0) {
        if (K < 4 || (K & (K - 1))) return 0;
        const int shared = levels_shared_by_samples(L);
        const int64_t level_bytes = ((int64_t)L.gp.T_mask + 1) * L.F * (L.tf16 ? 2 : 4);
        if (2 * shared >= L.gp.L) {
            if (K < 8 || level_bytes > L.l2_bytes) return 0;
            want = 4;
        } else {
            want = 4 * shared >= L.gp.L ? 2 : 1;
        }
    }
    if (want > K) want = K;
    int c = 1;
    while (2 * c <= want && 64 % (2 * c) == 0) c *= 2;
    return c;
}

// First level whose x-neighbour corner pairs are gathered as 16-byte
// blocks (gp.L: none; tables of 4-byte entries only).  By default the three
// finest levels (when a level's table exceeds one XCD's L2, whose misses
// scatter more: four, and at K >= 8 up to eight, which took the 8-view
// 1080p batch from 12.51 to 12.03 ms while 8 MiB levels at 720p and K = 8
// stayed within 0.2% and at K = 4 lost 2.6%; in rounds of one sample per
// ray, whose lanes are 64 rays whose samples lie apart on more levels: five,
// 1-3% faster at spacing 0.25 and K 4 to 16), among the hashed levels finer
// than a ray's sample spacing (coarser levels hand a ray's neighbouring
// samples the same lines, where a 4-byte gather is cheaper).  Measured against single-entry gathers
// on every level: the finest 2 to 4 levels were 2-15% faster at 720p (K 1 to
// 16, spacings 0.01 to 0.25, early termination or not) and 5-8% on the
// 8-view 1080p batch (8 MiB levels; 4 levels 1.5% faster there than 3),
// 1-5% slower only at K = 32 on a 4096-pixel-wide view; all hashed levels
// (or every level finer than the spacing) were slower on most.
static int render_block_from(const RenderLaunch &L)
{
    const int nl = L.gp.L;
    if (L.block_levels < 0) return nl;
    if (L.tf16 && L.F == 4) {
        // 8-byte entries: every hashed level, with 8 or more of them in
        // tables of at least 2^10 entries
        const int nd = L.gp.n_dense;
        if (L.block_levels > 0) return nl - L.block_levels > nd ? nl - L.block_levels : nd;
        return nl - nd >= 8 && L.gp.T_mask >= 1023u ? nd : nl;
    }
    if (!(L.tf16 && L.F == 2)) return nl;
    int lo = L.gp.n_dense;
    if (L.block_levels > 0) return nl - L.block_levels > lo ? nl - L.block_levels : lo;
    const int64_t level_bytes = ((int64_t)L.gp.T_mask + 1) * 4;
    const int kFinest = level_bytes > L.l2_bytes ? (L.rp.K >= 8 ? 8 : 4)
                        : render_chunk(L) == 1 ? 5 : 3;
    if (L.rp.K > 1) {
        const int shared = levels_shared_by_samples(L);
        if (shared > lo) lo = shared;
    }
    return nl - kFinest > lo ? nl - kFinest : (lo < nl ? lo : nl);
}

// Hashed levels per batch of gathers: 4 for entries of 8 or more bytes
// (F = 4 fp16 and up) when one batch then covers every hashed level of a
// query (at most 4), so a wave waits for its table once per tile instead of
// twice; else 2.  Measured at 720p with one query per pixel: the deployed
// grid (4 levels of 16 MiB) 5.5-8.6% faster with the Eq. 2 map, without it
// and without the MLP.  With 8 hashed levels, batches of 4 were 6% faster
// on 1 MiB levels without the MLP but 14% slower with the 2 x 8 MLP, 10%
// slower on 2^5-entry levels and 1.5% faster on 16 and 32 MiB levels, so 8
// levels keep batches of 2.  The batch changes only when loads are issued,
// never a result.
static int render_hash_batch(const RenderLaunch &L)
{
    const int eb = L.F * (L.tf16 ? 2 : 4);
    return eb >= 8 && L.gp.L - L.gp.n_dense <= 4 ? 4 : 2;
}

// Whether the waves claim the last units of their pools from the work
// counters (else every unit goes in the fixed order).  A claim is a
// device-scope atomic whose round trip costs about as much as a unit of 64
// samples over fewer than 8 levels without an MLP; there it is not hidden
// (K = 1, Tab. 3's frames with the MLP removed: L = 1..4 are 9% slower with
// claims), while with an MLP or 8 or more levels the balance they buy wins
// (3-6% at K = 1, 6% on the 1280x720 K = 8 frame, 15% on the 8-view batch).
static bool render_claims(const RenderLaunch &L)
{
    return L.nhid > 0 || L.gp.L >= 8;
}

// Grid size and tile order of a frame, given the blocks of its kernel that
// fit on one CU.
static void render_shape(const RenderLaunch &L, int resident, int64_t &blocks, int &stripe)
{
    const int R = kWave / L.rp.K;
    const TileShape ts = tile_shape(R, L.rp.views, L.rp.W, L.rp.H, 0);
    const int64_t want = ((int64_t)ts.n_tiles + kWavesPerBlock - 1) / kWavesPerBlock;
    // blocks resident on the whole device
    blocks = (int64_t)render_blocks_per_cu(L, resident) * L.cus;
    if (want < blocks) blocks = want;
    if (blocks > 8) blocks -= blocks % 8;
    if (blocks < 1) blocks = 1;
    stripe = render_stripe(L, ts, blocks);
}

// Blocks of one render kernel that fit on a CU, queried once per kernel.
template <int A, int B, bool C, int D, int E, int F_>
static int render_resident(bool queue)
{
    static std::atomic<int> cache{0}, cache_q{0};
    if (queue)
        return blocks_per_cu((const void *)render_queue_kernel<A, B, C, D, E, F_>, cache_q);
    return blocks_per_cu((const void *)render_kernel<A, B, C, D, E, F_>, cache);
}

#define MIXRT_RENDER_MATCH(a, b, c, d, e, f) \
    (L.tex == a && L.F == b && L.tf16 == c && L.nhid == f && (f == 0 || (L.in == d && L.hid == e)))

hipError_t launch_render(const RenderLaunch &L0, hipStream_t stream)
{
    RenderLaunch L = L0;
    L.gp.block_from = render_block_from(L);
    L.gp.hash_batch = render_hash_batch(L);
#define X(a, b, c, d, e, f)                                                                    \
    if (MIXRT_RENDER_MATCH(a, b, c, d, e, f)) {                                                \
        int64_t blocks;                                                                        \
        int stripe;                                                                            \
        const int chunk = render_chunk(L);                                                     \
        unsigned int *work = render_claims(L) ? L.work : nullptr;                              \
        render_shape(L, render_resident<a, b, c, d, e, f>(chunk > 0), blocks, stripe);         \
        if (chunk > 0)                                                                         \
            hipLaunchKernelGGL((render_queue_kernel<a, b, c, d, e, f>), dim3((unsigned)blocks), \
                               dim3(kBlock), 0, stream, L.rp, L.gp, L.weights, L.view_sh,      \
                               L.hid_w, stripe, chunk, work, L.out);                           \
        else                                                                                   \
            hipLaunchKernelGGL((render_kernel<a, b, c, d, e, f>), dim3((unsigned)blocks),      \
                               dim3(kBlock), 0, stream, L.rp, L.gp, L.weights, L.view_sh,      \
                               L.hid_w, stripe, work, L.out);                                  \
        return hipGetLastError();                                                              \
    }
    MIXRT_RENDER_VARIANTS(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t phase_cycles_read(uint64_t *out, bool reset)
{
#ifdef MIXRT_PHASE_TIMER
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpyFromSymbol(out, HIP_SYMBOL(phase_cycles), 8 * sizeof(uint64_t));
    if (e == hipSuccess && reset) {
        const unsigned long long zero[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        e = hipMemcpyToSymbol(HIP_SYMBOL(phase_cycles), zero, sizeof zero);
    }
    return e;
#else
    (void)out;
    (void)reset;
    return hipErrorNotSupported;
#endif
}

hipError_t render_launch_shape(const RenderLaunch &L, int *blocks, int *stripe, int *chunk,
                               int *block_from, int *hash_batch, int *claims)
{
    *block_from = render_block_from(L);
    *hash_batch = render_hash_batch(L);
    *claims = render_claims(L) ? 1 : 0;
#define X(a, b, c, d, e, f)                                                                    \
    if (MIXRT_RENDER_MATCH(a, b, c, d, e, f)) {                                                \
        int64_t nb;                                                                            \
        *chunk = render_chunk(L);                                                              \
        render_shape(L, render_resident<a, b, c, d, e, f>(*chunk > 0), nb, *stripe);          \
        *blocks = (int)nb;                                                                     \
        return hipSuccess;                                                                     \
    }
    MIXRT_RENDER_VARIANTS(X)
#undef X
    return hipErrorInvalidValue;
}

}  // namespace mixrt
