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
