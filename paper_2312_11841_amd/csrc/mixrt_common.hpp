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
