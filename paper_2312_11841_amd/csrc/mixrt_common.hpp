// Launch geometry shared by the kernels of mixrt_render.hip and
// mixrt_stages.hip.
#pragma once

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

// Blocks of `fn` resident on the whole device at once (at least one per CU).
inline int resident_blocks(const void *fn, int cus)
{
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, 0) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    return per_cu * cus;
}

}  // namespace mixrt
