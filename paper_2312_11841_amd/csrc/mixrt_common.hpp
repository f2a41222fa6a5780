// Launch geometry shared by the kernels of mixrt_render.hip and
// mixrt_stages.hip.
#pragma once

#include <atomic>

#include "mixrt_device.hpp"

namespace mixrt {


inline constexpr int kBlock = 256;             // 4 waves
inline constexpr int kWavesPerBlock = kBlock / kWave;

// Block -> logical block so that each XCD (blocks are dealt round-robin to
// the 8 XCDs) works on a contiguous range of tiles and shares its L2.
__device__ __forceinline__ int xcd_logical_block(int b, int nb)
{
    if (nb % 8 != 0) return b;
    return (b & 7) * (nb >> 3) + (b >> 3);
}

// Work distribution for the persistent render kernels.  The units (tiles,
// or runs of tiles) are split into P pools, one per XCD when the grid is a
// multiple of 8 blocks (else one pool): unit u of pool p is the global unit
// (u / Wp) * total + p * Wp + u % Wp, with Wp = total / P waves per pool,
// so that an XCD's units in flight are a compact run of the tile order.
//
// Wave j of pool p takes units j, j + Wp, j + 2 Wp, ... for its first S
// rounds (85% of the rounds a static split gives it, at most 16); the rest
// of the pool's units are handed out in order from counters, so that waves
// that run faster take more of them instead of idling while the slowest
// finish a fixed share, and the units an XCD works on at once stay one
// compact run however far its waves have drifted apart.  A pool has 4
// counters, one per wave slot of a block, each handing out every fourth
// unit: a device-scope atomic on one address is performed at the memory
// side one at a time (about 11 ns apart), so one counter per pool would
// queue its waves' claims.  A wave claims its next unit while it runs the
// current one's MLP, so the claim's latency is hidden.
//
// Without counters (a null pointer) every unit goes in the fixed order, the
// static split's last round partial.
//
// The counters live in device memory the caller provides (kWorkWords
// 32-bit words, zero before a launch): claim counter c of pool p at word
// (p * kWorkSub + c) * kWorkStride, the count of the pool's finished blocks
// at (kWorkPools * kWorkSub + p) * kWorkStride, each in its own 256-byte
// block.  The last block of a pool to finish sets the pool's words back to
// zero, so a buffer is ready for the next launch on the same stream.  Two
// launches that run at the same time must not share a buffer.
inline constexpr int kWorkStride = 64;
inline constexpr int kWorkPools = 8;
inline constexpr int kWorkSub = 4;
inline constexpr int kWorkWords = (kWorkSub + 1) * kWorkPools * kWorkStride;
inline constexpr int kWorkStaticPct = 85;   // of a wave's static rounds taken statically
inline constexpr int kWorkStaticMax = 16;   // at most this many

struct WorkPools {
    unsigned int *ctr;
    int nU;                  // units
    int P, pool, Wp, total, j, S, sub;
    int r;                   // static rounds taken
    int Sc;                  // S with counters, -1 without (no claim is due)
    bool want;               // the next claim is still to be issued
    int end;                 // the units this wave's pool hands out
    unsigned int inv;        // ceil(2^32 / Wp), for dividing by Wp
    unsigned int pending;    // lane 0: the claim in flight

    __device__ __forceinline__ WorkPools(unsigned int *c, int n_units, int lane)
        : ctr(c), nU(n_units), r(0), want(false), pending(0u)
    {
        const int nb = (int)gridDim.x;
        total = nb * kWavesPerBlock;
        P = nb % 8 == 0 ? 8 : 1;
        pool = P == 8 ? (int)(blockIdx.x & 7) : 0;
        Wp = total / P;
        // this wave's index in its pool (blocks of a pool: b = pool + 8 i)
        j = (P == 8 ? (int)(blockIdx.x >> 3) : (int)blockIdx.x) * kWavesPerBlock +
            (int)__builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
        sub = j & (kWorkSub - 1);
        const int full = n_units / total;
        int rest = n_units - full * total - pool * Wp;
        rest = rest < 0 ? 0 : rest > Wp ? Wp : rest;
        end = full * Wp + rest;
        inv = __builtin_amdgcn_readfirstlane(0xffffffffu / (unsigned int)Wp + 1u);
        if (ctr) {
            S = (full * kWorkStaticPct) / 100;
            if (S > kWorkStaticMax) S = kWorkStaticMax;
            if (S == 0 && full > 0) S = 1;
            if (S == 0) pending = claim(lane);
            Sc = S;
        } else {
            // no counters: every unit in the fixed order, the last round
            // partial, and no unit to claim after it
            S = (n_units + total - 1) / total;
            Sc = -1;
            end = 0;
        }
    }
    // issues the claim of the wave's next counted unit, if it is due.  The
    // kernels call this once their gathers of a unit have returned (memory
    // results come back in order, so the first wait for a load issued after
    // the claim also waits for the claim): the claim then overlaps the MLP
    // and compositing, not the next unit's loads
    __device__ __forceinline__ void prefetch(int lane)
    {
        if (want) {
            pending = claim(lane);
            want = false;
        }
    }
    // lane 0 claims the next counted unit of this wave's pool; the value is
    // read later, so the claim is in flight meanwhile
    __device__ __forceinline__ unsigned int claim(int lane) const
    {
        unsigned int u = 0;
        if (lane == 0) u = atomicAdd(&ctr[(pool * kWorkSub + sub) * kWorkStride], 1u);
        return u;
    }
    // the next unit of this wave, or -1 when its pool is spent
    __device__ __forceinline__ int take(int lane)
    {
        if (__builtin_expect(r < S, 1)) {
            const int t = r * total + pool * Wp + j;
            if (t >= nU) return -1;   // the fixed order's partial last round
            want = ++r == Sc;
            return t;
        }
        prefetch(lane);
        const int c = (int)__builtin_amdgcn_readfirstlane(pending);
        const int d = S * Wp + c * kWorkSub + sub;
        if (d >= end) return -1;
        want = true;
        // pool unit d is unit (d / Wp) * total + pool * Wp + d % Wp; the
        // quotient from the reciprocal is exact or one too large (d < 2^31)
        unsigned int q = __umulhi((unsigned int)d, inv);
        if (q * (unsigned int)Wp > (unsigned int)d) --q;
        return (int)q * (total - Wp) + pool * Wp + d;
    }
    // after the wave's last take, at the end of the kernel (every wave of
    // the block gets here): the block counts itself done in its pool, and
    // the pool's last block clears the pool's counters for the next launch
    __device__ __forceinline__ void finish() const
    {
        if (!ctr) return;
        __syncthreads();
        if (threadIdx.x == 0) {
            unsigned int *done = &ctr[(kWorkPools * kWorkSub + pool) * kWorkStride];
            const unsigned int d = atomicAdd(done, 1u);
            if (d == (unsigned int)((int)gridDim.x / P) - 1u) {
                for (int i = 0; i < kWorkSub; ++i)
                    atomicExch(&ctr[(pool * kWorkSub + i) * kWorkStride], 0u);
                atomicExch(done, 0u);
            }
        }
    }
};

// A tile's R = 64/K rays cover a block of pixels, RW x RH with RW >= 4 RH,
// when R is a power of two (8 rays: 8 x 1; 64 rays: 16 x 4), else one row
// segment.  With one sample per ray the block puts nearby pixels in one wave,
// so its gathers share more cache lines (K = 1: 10-16% faster than a row of
// 64); with 8 samples per ray a row of 8 measured best.  Tiles never cross a
// row or view boundary.
//
// Tile order: tiles are numbered view by view; inside a view, in vertical
// stripes `stripe` tiles wide (the last one narrower), each stripe row by
// row.  A stripe as wide as the view is plain row-major order.  Waves take
// tiles in this order, so consecutive runs of tiles (the tiles one XCD works
// on at once) are compact blocks of pixels `stripe` tiles wide.
struct TileShape {
    int RW, RH, tiles_x, tiles_y, per_view, n_tiles, stripe;
};

__host__ __device__ inline TileShape tile_shape(int R, int views, int W, int H, int stripe)
{
    TileShape t;
    t.RH = 1;
    if ((R & (R - 1)) == 0)
        while (t.RH * t.RH * 16 <= R) t.RH *= 2;
    t.RW = R / t.RH;
    t.tiles_x = (W + t.RW - 1) / t.RW;
    t.tiles_y = (H + t.RH - 1) / t.RH;
    t.per_view = t.tiles_x * t.tiles_y;
    t.n_tiles = views * t.per_view;
    t.stripe = (stripe < 1 || stripe > t.tiles_x) ? t.tiles_x : stripe;
    return t;
}

struct TilePos {
    int view, tx, ty;
};

// The s-th tile of the order above (0 <= s < n_tiles).
__host__ __device__ inline TilePos tile_at(const TileShape &t, int s)
{
    TilePos p;
    p.view = s / t.per_view;
    int rem = s - p.view * t.per_view;
    const int band = t.stripe * t.tiles_y;   // tiles in one full-width stripe
    const int b = rem / band;
    rem -= b * band;
    const int x0 = b * t.stripe;
    const int w = t.tiles_x - x0 < t.stripe ? t.tiles_x - x0 : t.stripe;
    p.ty = rem / w;
    p.tx = x0 + rem - p.ty * w;
    return p;
}

__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Blocks of `fn` (kBlock threads) resident on one CU at once, at least 1;
// queried once per kernel and kept in `cache` (the value depends only on the
// kernel), so concurrent first calls at worst query twice.
inline int blocks_per_cu(const void *fn, std::atomic<int> &cache)
{
    int per_cu = cache.load(std::memory_order_relaxed);
    if (per_cu > 0) return per_cu;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, 0) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    cache.store(per_cu, std::memory_order_relaxed);
    return per_cu;
}

}  // namespace mixrt
