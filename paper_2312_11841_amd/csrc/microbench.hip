// Roofline microbenchmarks for gfx950, used to calibrate the rendering
// kernel's measured bounds (not part of the rendering path):
//   - gather: random or coalesced loads of 4/8/16 bytes per lane from a
//     table of a given size (the access pattern of hash-grid lookups), which
//     measures the achievable gather rate by working set (L1/L2/MALL/HBM);
//   - copy:   a streaming copy (HBM bandwidth, reads and writes);
//   - read:   a streaming read (HBM read bandwidth, the hot path's mix);
//   - mfma:   a dependent-free fp16 16x16x32 MFMA loop (matrix-core peak).
// Entry points launch on the given stream and return hipError_t codes; the
// caller times them with events on that stream.
#include <string.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cmath>

#include "mixrt_common.hpp"
#include "mixrt_microbench.h"

static_assert(MIXRT_MB_WORK_WORDS == mixrt::kWorkWords, "replay work counters");

namespace {

constexpr int kBlock = 256;

template <int W>
struct Vec;
template <>
struct Vec<4> {
    typedef uint32_t T;
    static __device__ __forceinline__ uint32_t fold(T v) { return v; }
};
template <>
struct Vec<8> {
    typedef uint2 T;
    static __device__ __forceinline__ uint32_t fold(T v) { return v.x ^ v.y; }
};
template <>
struct Vec<16> {
    typedef uint4 T;
    static __device__ __forceinline__ uint32_t fold(T v) { return v.x ^ v.y ^ v.z ^ v.w; }
};

// Each lane walks its own xorshift stream; per iteration it issues NL
// independent loads (all issued before any is consumed).  pattern 0: a
// random W-byte element per load; pattern 1: every lane of the wave loads
// the same element (one cache line per instruction).
template <int W, int NL>
__global__ __launch_bounds__(kBlock) void gather_kernel(const char *__restrict__ table,
                                                        uint32_t n_elems_mask, int iters,
                                                        int pattern, uint32_t *__restrict__ sink)
{
    typedef typename Vec<W>::T T;
    const uint32_t gid = blockIdx.x * kBlock + threadIdx.x;
    uint32_t x = gid * 2654435761u + 12345u;
    const uint32_t wave_seed = (gid / 64u) * 2246822519u + 777u;
    uint32_t acc = 0;
    for (int it = 0; it < iters; ++it) {
        uint32_t off[NL];
#pragma unroll
        for (int q = 0; q < NL; ++q) {
            x ^= x << 13;
            x ^= x >> 17;
            x ^= x << 5;
            const uint32_t r = pattern ? (wave_seed + (uint32_t)(it * NL + q) * 40503u) : x;
            off[q] = (r & n_elems_mask) * (uint32_t)W;
        }
        T v[NL];
#pragma unroll
        for (int q = 0; q < NL; ++q)
            v[q] = *(const T *)(table + off[q]);
#pragma unroll
        for (int q = 0; q < NL; ++q)
            acc ^= Vec<W>::fold(v[q]);
    }
    sink[gid] = acc;
}

// Gathers whose 64 lanes touch exactly D distinct 128-byte lines per
// instruction (D divides 64), 64/D lanes per line: lanes j*64/D .. (j+1)*64/D
// - 1 on line j when `adjacent`, else lane l on line l mod D; within a line
// the lanes take consecutive W-byte words.  Each iteration issues 8
// independent loads on fresh pseudo-random line sets of a table of n_lines
// lines (a power of two).  The time per instruction tells how the vector L1
// charges a gather: by lanes, by distinct lines, or by lanes per line.
template <int W>
__global__ __launch_bounds__(kBlock) void lines_kernel(const char *__restrict__ table,
                                                       uint32_t line_mask, int iters, int D,
                                                       int adjacent, uint32_t *__restrict__ sink)
{
    typedef typename Vec<W>::T T;
    const int lane = threadIdx.x & 63;
    const uint32_t gw = blockIdx.x * (kBlock / 64) + threadIdx.x / 64;
    const int per = 64 / D;
    const uint32_t j = (uint32_t)(adjacent ? lane / per : lane % D);
    const uint32_t q = (uint32_t)(adjacent ? lane % per : lane / D);
    const uint32_t within = (q * (uint32_t)W) & (128u - (uint32_t)W);
    uint32_t base = gw * 2654435761u + 12345u, acc = 0;
    for (int it = 0; it < iters; ++it) {
        T v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const uint32_t b = (base + (uint32_t)u * 0x9E3779B9u) >> 7;
            const uint32_t line = (b * 64u + j * 97u) & line_mask;
            v[u] = *(const T *)(table + (size_t)line * 128u + within);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) acc ^= Vec<W>::fold(v[u]);
        base = base * 1664525u + 1013904223u;
    }
    sink[blockIdx.x * kBlock + threadIdx.x] = acc;
}

__global__ __launch_bounds__(kBlock) void copy_kernel(const uint4 *__restrict__ src,
                                                      uint4 *__restrict__ dst, uint64_t n)
{
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride)
        dst[i] = src[i];
}

// Grid-stride read of n 16-byte elements, four independent loads per thread
// in flight per iteration; each thread writes one word (the XOR of what it
// read) so the loads stay live.
__global__ __launch_bounds__(kBlock) void read_kernel(const uint4 *__restrict__ src, uint64_t n,
                                                      uint32_t *__restrict__ sink)
{
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    uint32_t acc = 0;
    for (; i + 3 * stride < n; i += 4 * stride) {
        const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride],
                    d = src[i + 3 * stride];
        acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^
               d.z ^ d.w;
    }
    for (; i < n; i += stride) {
        const uint4 a = src[i];
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    sink[(uint64_t)blockIdx.x * kBlock + threadIdx.x] = acc;
}

// Mixed read/write stream in the MLP stage's pattern: each wave takes tiles
// of 64 rows of `in_chunks` 16-byte chunks (read coalesced, lane l taking
// chunks l, l + 64, ...) and writes one 16-byte chunk per row (64 per tile),
// so reads and writes keep the stage's ratio (96 B in, 16 B out per row for
// 48 fp16 inputs).  Loads and stores are non-temporal like the stage's.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int IN_CHUNKS>
__global__ __launch_bounds__(kBlock) void rowstream_kernel(const u32x4 *__restrict__ src,
                                                           u32x4 *__restrict__ dst,
                                                           int64_t n_tiles)
{
    const int lane = threadIdx.x & 63;
    const int64_t total = (int64_t)gridDim.x * (kBlock / 64);
    for (int64_t t = (int64_t)blockIdx.x * (kBlock / 64) + threadIdx.x / 64; t < n_tiles;
         t += total) {
        const u32x4 *s = src + t * 64 * IN_CHUNKS;
        u32x4 v[IN_CHUNKS];
#pragma unroll
        for (int c = 0; c < IN_CHUNKS; ++c) v[c] = __builtin_nontemporal_load(s + c * 64 + lane);
        u32x4 a = v[0];
#pragma unroll
        for (int c = 1; c < IN_CHUNKS; ++c) a ^= v[c];
        __builtin_nontemporal_store(a, dst + t * 64 + lane);
    }
}

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

// 8 independent accumulators per wave, so consecutive MFMAs do not depend on
// each other.
__global__ __launch_bounds__(kBlock) void mfma_kernel(int iters, float *__restrict__ out)
{
    const int lane = threadIdx.x & 63;
    h8 a, b;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        a[j] = (_Float16)(0.001f * (lane + j));
        b[j] = (_Float16)(0.002f * (lane - j));
    }
    f4 acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
            acc[u] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc[u], 0, 0, 0);
    }
    f4 s = acc[0];
#pragma unroll
    for (int u = 1; u < 8; ++u) s += acc[u];
    out[blockIdx.x * kBlock + threadIdx.x] = s[0] + s[1] + s[2] + s[3];
}

// ---------------------------------------------------------------------------
// Gather replay: the hash-grid loads of one frame, in the render kernel's
// order and nothing else.  Same persistent grid, work distribution (the
// per-XCD pools: a static start, then runs claimed from the counters) and
// tile order (stripe) as the render kernel; a lane takes the
// same sample of the same tile, reads that sample's position from the frame's
// ray-setup output, and issues the same loads in the same batches (dense
// levels as x-neighbour pairs, hashed levels of 4- or 8-byte entries from
// block_from on as 16-byte blocks per x-neighbour pair).  The corner entries'
// words are XOR-folded into one word per lane (no fp16 conversion, no interpolation,
// no MLP, no compositing), so the kernel's time is the floor that this exact
// access stream, plus the address arithmetic that produces it, sets.  MODE 1
// drops the loads and folds the offsets instead (the address arithmetic
// alone).
// ---------------------------------------------------------------------------
template <uint32_t EB>
struct RawEntry;
template <> struct RawEntry<4> {
    static __device__ __forceinline__ uint32_t one(const char *t, uint32_t o)
    {
        return *(const uint32_t *)(t + o);
    }
    static __device__ __forceinline__ uint32_t pair(const char *t, uint32_t o)
    {
        const uint64_t v = *(const mixrt::u64a4 *)(t + o);
        return (uint32_t)v ^ (uint32_t)(v >> 32);
    }
};
template <> struct RawEntry<8> {
    static __device__ __forceinline__ uint32_t one(const char *t, uint32_t o)
    {
        const uint2 v = *(const uint2 *)(t + o);
        return v.x ^ v.y;
    }
    static __device__ __forceinline__ uint32_t pair(const char *t, uint32_t o)
    {
        const unsigned __int128 v = *(const mixrt::u128a8 *)(t + o);
        return (uint32_t)v ^ (uint32_t)(v >> 32) ^ (uint32_t)(v >> 64) ^ (uint32_t)(v >> 96);
    }
};
template <> struct RawEntry<16> {
    static __device__ __forceinline__ uint32_t one(const char *t, uint32_t o)
    {
        const uint4 v = *(const uint4 *)(t + o);
        return v.x ^ v.y ^ v.z ^ v.w;
    }
    static __device__ __forceinline__ uint32_t pair(const char *t, uint32_t o)
    {
        return one(t, o) ^ one(t, o + 16u);
    }
};

template <uint32_t EB, int G, bool DENSE, int MODE, bool BLOCKS = false>
__device__ __forceinline__ uint32_t replay_group(const mixrt::GridParams &gp, int l0, float x0,
                                                 float x1, float x2)
{
    mixrt::LevelSetup s[G];
#pragma unroll
    for (int g = 0; g < G; ++g)
        mixrt::level_setup<EB, true>(gp, l0 + g, DENSE, x0, x1, x2, s[g]);
    // hashed levels with 4- or 8-byte entries from block_from on: the
    // render's block loads (one aligned 16-byte block per x-neighbour pair,
    // the x + 1 entries loaded apart where the voxel straddles two blocks),
    // and the two entries' words picked
    constexpr bool kBlocks = BLOCKS && !DENSE && (EB == 4 || EB == 8);
    uint32_t v[G][8];
    uint4 blk[G][4];
    uint32_t far[G][4];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const char *t = (const char *)gp.table + (size_t)(l0 + g) * ((size_t)gp.T_mask + 1) * EB;
        if (kBlocks && MODE == 0) {
            const bool straddle = (s[g].off[0] ^ s[g].off[1]) >= 16u;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                blk[g][q] = *(const uint4 *)(t + (s[g].off[2 * q] & ~15u));
                far[g][q] = 0u;
            }
            if (straddle) {
#pragma unroll
                for (int q = 0; q < 4; ++q) far[g][q] = RawEntry<EB>::one(t, s[g].off[2 * q + 1]);
            }
            continue;
        }
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            if (DENSE && (b & 1)) continue;   // a dense pair covers corners b and b + 1
            if (MODE == 1)
                v[g][b] = s[g].off[b];
            else
                v[g][b] = DENSE ? RawEntry<EB>::pair(t, s[g].off[b]) : RawEntry<EB>::one(t, s[g].off[b]);
        }
    }
    uint32_t acc = 0;
#pragma unroll
    for (int g = 0; g < G; ++g) {
        if (kBlocks && MODE == 0) {
            const bool straddle = (s[g].off[0] ^ s[g].off[1]) >= 16u;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if constexpr (EB == 4) {
                    acc ^= mixrt::block_word(blk[g][q], s[g].off[2 * q]);
                    acc ^= straddle ? far[g][q] : mixrt::block_word(blk[g][q], s[g].off[2 * q + 1]);
                } else {
                    // 8-byte entries: the pair's two entries are the block's halves
                    const uint4 b = blk[g][q];
                    acc ^= straddle ? (((s[g].off[2 * q] & 8u) ? (b.z ^ b.w) : (b.x ^ b.y)) ^ far[g][q])
                                    : (b.x ^ b.y ^ b.z ^ b.w);
                }
            }
            continue;
        }
#pragma unroll
        for (int b = 0; b < 8; ++b)
            if (!(DENSE && (b & 1))) acc ^= v[g][b];
    }
    return acc;
}

template <uint32_t EB, int MODE>
__global__ __launch_bounds__(kBlock) void replay_kernel(const float *__restrict__ x,
                                                        const int32_t *__restrict__ hit, int views,
                                                        int W, int H, int K, int stripe, int C,
                                                        mixrt::GridParams gp,
                                                        unsigned int *__restrict__ work,
                                                        uint32_t *__restrict__ sink)
{
    constexpr int kGroup = 2;
    const int lane = threadIdx.x & 63;
    const int R = 64 / K;
    const mixrt::TileShape ts = mixrt::tile_shape(R, views, W, H, stripe);
    const int L = gp.L, n_dense = gp.n_dense;
    // C = 0: one tile per step, lane r K + k on sample k of ray r (the tile
    // path).  C > 0: the early-termination path's order when no ray stops
    // and every ray hits: runs of B = K/C tiles, one round per C samples,
    // lane s C + j on sample c C + j of the run's ray s.
    const int B = C > 0 && K / C > 1 ? K / C : 1;
    const int rounds = C > 0 ? (K + C - 1) / C : 1;
    const int Cl = C > 0 ? C : K;
    const int sl = lane / Cl, j = lane - sl * Cl;
    const int t_in_run = C > 0 ? sl / R : 0, r_loc = C > 0 ? sl - t_in_run * R : lane / K;
    uint32_t acc = 0;
    // runs from the render kernels' per-XCD pools (work null: all in the
    // fixed order); the claim of a wave's next run goes out once the current
    // run's first round of loads is done
    mixrt::WorkPools pools(work, (ts.n_tiles + B - 1) / B, lane);
    for (;;) {
    const int run = pools.take(lane);
    if (run < 0) break;
    for (int c = 0; c < rounds; ++c) {
        if (c > 0) pools.prefetch(lane);
        const int64_t tile64 = (int64_t)run * B + t_in_run;
        const int k = C > 0 ? c * C + j : lane - r_loc * K;
        if (t_in_run >= B || tile64 >= ts.n_tiles || k >= K || lane >= (C > 0 ? 64 : R * K))
            continue;
        const mixrt::TilePos tp = mixrt::tile_at(ts, (int)tile64);
        const int i0 = tp.tx * ts.RW, j0 = tp.ty * ts.RH;
        const int dy = r_loc / ts.RW, dx = r_loc - dy * ts.RW;
        const bool valid = r_loc < R && i0 + dx < W && j0 + dy < H;
        if (!valid) continue;
        const int ray = (tp.view * H + j0 + dy) * W + i0 + dx;
        if (!hit[ray]) continue;
        const float *p = x + ((size_t)ray * K + k) * 3;
        // positions into [0, 1] (NaN to 0), which level_setup's in-unit form
        // needs to keep every corner inside its level
        const float x0 = p[0] >= 0.0f ? fminf(p[0], 1.0f) : 0.0f;
        const float x1 = p[1] >= 0.0f ? fminf(p[1], 1.0f) : 0.0f;
        const float x2 = p[2] >= 0.0f ? fminf(p[2], 1.0f) : 0.0f;
        int l = 0;
        for (; l + kGroup <= n_dense; l += kGroup) acc ^= replay_group<EB, kGroup, true, MODE>(gp, l, x0, x1, x2);
        for (; l < n_dense; ++l) acc ^= replay_group<EB, 1, true, MODE>(gp, l, x0, x1, x2);
        const int lb = (EB == 4 || EB == 8) && gp.block_from < L ? max(gp.block_from, l) : L;
        // 8-byte entries: 4 levels per batch without blocks when hash_batch
        // asks for it, else pairs of levels, with blocks from block_from on,
        // as the render batches them
        if (EB >= 8 && gp.hash_batch >= 4 && lb == L)
            for (; l + 4 <= lb; l += 4) acc ^= replay_group<EB, 4, false, MODE>(gp, l, x0, x1, x2);
        for (; l + kGroup <= lb; l += kGroup) acc ^= replay_group<EB, kGroup, false, MODE>(gp, l, x0, x1, x2);
        for (; l < lb; ++l) acc ^= replay_group<EB, 1, false, MODE>(gp, l, x0, x1, x2);
        if (EB == 8)
            for (; l + kGroup <= L; l += kGroup) acc ^= replay_group<EB, kGroup, false, MODE, true>(gp, l, x0, x1, x2);
        for (; l < L; ++l) acc ^= replay_group<EB, 1, false, MODE, true>(gp, l, x0, x1, x2);
    }
    pools.prefetch(lane);
    }
    pools.finish();
    sink[(size_t)blockIdx.x * kBlock + threadIdx.x] = acc;
}

}  // namespace

extern "C" {

int mixrt_mb_gather_replay(const float *x, const int32_t *hit, int32_t views, int32_t W,
                           int32_t H, int32_t K, const void *table, int32_t L, int32_t log2_T,
                           int32_t entry_bytes, const int32_t *N, int32_t tile_stripe,
                           int32_t chunk, int32_t block_from, int32_t hash_batch,
                           int32_t mode, int32_t blocks, uint32_t *work, uint32_t *sink,
                           void *stream)
{
    if (!x || !hit || !table || !N || !sink) return hipErrorInvalidValue;
    if (chunk < 0 || chunk > K || (chunk > 0 && (64 % chunk != 0 || (chunk & (chunk - 1)))))
        return hipErrorInvalidValue;
    if (views < 1 || W < 1 || H < 1 || (int64_t)views * H * W >= ((int64_t)1 << 31))
        return hipErrorInvalidValue;
    if (K < 1 || K > 64 || L < 1 || L > mixrt::kMaxLevels || log2_T < 4 || log2_T > 26)
        return hipErrorInvalidValue;
    if (entry_bytes != 4 && entry_bytes != 8 && entry_bytes != 16) return hipErrorInvalidValue;
    if ((mode != 0 && mode != 1) || blocks < 1) return hipErrorInvalidValue;
    if (hash_batch != 2 && hash_batch != 4) return hipErrorInvalidValue;
    if (((uintptr_t)table & 15) != 0) return hipErrorInvalidValue;
    mixrt::GridParams gp;
    memset(&gp, 0, sizeof gp);
    gp.table = table;
    gp.log2_T = (uint32_t)log2_T;
    gp.T_mask = (uint32_t)((1u << log2_T) - 1u);
    gp.L = L;
    gp.block_from = block_from < 0 ? 0 : block_from > L ? L : block_from;
    gp.hash_batch = hash_batch;
    const uint64_t T = 1ull << log2_T;
    for (int l = 0; l < L; ++l) {
        if (N[l] < 1 || N[l] > (1 << 20) || (l > 0 && N[l] < N[l - 1])) return hipErrorInvalidValue;
        gp.N[l] = (uint32_t)N[l];
        gp.Nf[l] = (float)N[l];
        gp.Ntop[l] = (float)(N[l] - 1);
        const uint64_t side = (uint64_t)N[l] + 1;
        if (side * side * side <= T) {
            gp.dense_mask |= 1u << l;
            gp.n_dense = l + 1;
        }
    }
    hipStream_t s = (hipStream_t)stream;
#define RP(EB, M)                                                                                \
    hipLaunchKernelGGL((replay_kernel<EB, M>), dim3(blocks), dim3(kBlock), 0, s, x, hit, views, \
                       W, H, K, tile_stripe, chunk, gp, work, sink)
    if (mode == 0) {
        if (entry_bytes == 4) RP(4, 0);
        else if (entry_bytes == 8) RP(8, 0);
        else RP(16, 0);
    } else {
        if (entry_bytes == 4) RP(4, 1);
        else if (entry_bytes == 8) RP(8, 1);
        else RP(16, 1);
    }
#undef RP
    return hipGetLastError();
}

int mixrt_mb_gather(const void *table, uint64_t table_bytes, int width, int loads_per_iter,
                    int iters, int pattern, int blocks, uint32_t *sink, void *stream)
{
    if (!table || !sink || blocks < 1 || iters < 1) return hipErrorInvalidValue;
    if (width != 4 && width != 8 && width != 16) return hipErrorInvalidValue;
    if (loads_per_iter != 1 && loads_per_iter != 8) return hipErrorInvalidValue;
    const uint64_t n = table_bytes / (uint64_t)width;
    if (n == 0 || (n & (n - 1)) || n > (1ull << 32)) return hipErrorInvalidValue;
    const uint32_t mask = (uint32_t)(n - 1);
    hipStream_t s = (hipStream_t)stream;
    const char *t = (const char *)table;
#define G(W, NL)                                                                              \
    hipLaunchKernelGGL((gather_kernel<W, NL>), dim3(blocks), dim3(kBlock), 0, s, t, mask, iters, \
                       pattern, sink)
    if (loads_per_iter == 8) {
        if (width == 4) G(4, 8);
        else if (width == 8) G(8, 8);
        else G(16, 8);
    } else {
        if (width == 4) G(4, 1);
        else if (width == 8) G(8, 1);
        else G(16, 1);
    }
#undef G
    return hipGetLastError();
}

int mixrt_mb_gather_lines(const void *table, uint64_t table_bytes, int width, int lines,
                          int adjacent, int iters, int blocks, uint32_t *sink, void *stream)
{
    if (!table || !sink || blocks < 1 || iters < 1) return hipErrorInvalidValue;
    if (width != 4 && width != 8 && width != 16) return hipErrorInvalidValue;
    if (lines < 1 || lines > 64 || 64 % lines != 0) return hipErrorInvalidValue;
    const uint64_t n = table_bytes / 128u;
    if (n == 0 || (n & (n - 1)) || n > (1ull << 31) || n * 128u != table_bytes)
        return hipErrorInvalidValue;
    const uint32_t mask = (uint32_t)(n - 1);
    hipStream_t s = (hipStream_t)stream;
    const char *t = (const char *)table;
#define LK(W)                                                                                   \
    hipLaunchKernelGGL((lines_kernel<W>), dim3(blocks), dim3(kBlock), 0, s, t, mask, iters, lines, \
                       adjacent, sink)
    if (width == 4) LK(4);
    else if (width == 8) LK(8);
    else LK(16);
#undef LK
    return hipGetLastError();
}

int mixrt_mb_copy(const void *src, void *dst, uint64_t bytes, int blocks, void *stream)
{
    if (!src || !dst || (bytes & 15) || blocks < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(kBlock), 0, (hipStream_t)stream,
                       (const uint4 *)src, (uint4 *)dst, bytes / 16);
    return hipGetLastError();
}

int mixrt_mb_read(const void *src, uint64_t bytes, int blocks, uint32_t *sink, void *stream)
{
    if (!src || !sink || (bytes & 15) || blocks < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(read_kernel, dim3(blocks), dim3(kBlock), 0, (hipStream_t)stream,
                       (const uint4 *)src, bytes / 16, sink);
    return hipGetLastError();
}

int mixrt_mb_rowstream(const void *src, void *dst, int64_t rows, int in_bytes, int blocks,
                       void *stream)
{
    if (!src || !dst || blocks < 1 || rows < 0 || rows % 64) return hipErrorInvalidValue;
    if (((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return hipErrorInvalidValue;
    const int64_t tiles = rows / 64;
    hipStream_t s = (hipStream_t)stream;
#define RS(C)                                                                                   \
    hipLaunchKernelGGL((rowstream_kernel<C>), dim3(blocks), dim3(kBlock), 0, s,                  \
                       (const u32x4 *)src, (u32x4 *)dst, tiles)
    switch (in_bytes) {
    case 32: RS(2); break;
    case 64: RS(4); break;
    case 96: RS(6); break;
    default: return hipErrorInvalidValue;
    }
#undef RS
    return hipGetLastError();
}

int mixrt_mb_mfma(int iters, int blocks, float *out, void *stream)
{
    if (!out || blocks < 1 || iters < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(mfma_kernel, dim3(blocks), dim3(kBlock), 0, (hipStream_t)stream, iters,
                       out);
    return hipGetLastError();
}

int mixrt_mb_device_info(int device, int *clock_khz, int *mem_clock_khz, int *cus,
                         int *l2_bytes, char *arch, int cap)
{
    hipDeviceProp_t p;
    const hipError_t e = hipGetDeviceProperties(&p, device);
    if (e != hipSuccess) return (int)e;
    if (clock_khz) *clock_khz = p.clockRate;
    if (mem_clock_khz) *mem_clock_khz = p.memoryClockRate;
    if (cus) *cus = p.multiProcessorCount;
    if (l2_bytes) *l2_bytes = p.l2CacheSize;
    if (arch && cap > 0) {
        strncpy(arch, p.gcnArchName, (size_t)cap - 1);
        arch[cap - 1] = 0;
    }
    return 0;
}

}  // extern "C"
