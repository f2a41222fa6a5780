// Internal interface between the C ABI (mixrt_api.cpp) and the kernels
// (mixrt_render.hip, mixrt_stages.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <type_traits>

#include "mixrt_device.hpp"

namespace mixrt {

// Texture kinds the kernels are built for: (element type, displacement form,
// SH degree of Eq. 2's vector form).
enum TexId {
    kTexF32Ray,
    kTexF16Ray,
    kTexU8Ray,
    kTexF32Vec3D1,
    kTexF16Vec3D2,
    kTexU8Vec3D2,
    kTexNone,
    kTexF32Vec3,   // Eq. 2 as printed, SH degree 0..3 at run time
    kTexF16Vec3,
    kTexU8Vec3,
};

template <int ID>
struct TexOf;
template <> struct TexOf<kTexF32Ray> { typedef TexKind<float, kDispAlongRay> type; };
template <> struct TexOf<kTexF16Ray> { typedef TexKind<_Float16, kDispAlongRay> type; };
template <> struct TexOf<kTexU8Ray> { typedef TexKind<uint8_t, kDispAlongRay> type; };
template <> struct TexOf<kTexF32Vec3D1> { typedef TexKind<float, kDispShVec3, 1> type; };
template <> struct TexOf<kTexF16Vec3D2> { typedef TexKind<_Float16, kDispShVec3, 2> type; };
template <> struct TexOf<kTexU8Vec3D2> { typedef TexKind<uint8_t, kDispShVec3, 2> type; };
template <> struct TexOf<kTexNone> { typedef TexKind<float, kDispNone> type; };
template <> struct TexOf<kTexF32Vec3> { typedef TexKind<float, kDispShVec3, -1> type; };
template <> struct TexOf<kTexF16Vec3> { typedef TexKind<_Float16, kDispShVec3, -1> type; };
template <> struct TexOf<kTexU8Vec3> { typedef TexKind<uint8_t, kDispShVec3, -1> type; };

// dtype: 0 f32, 1 f16, 2 u8 (mixrt_dtype); mode: mixrt_disp_mode.  -1 when
// no kernel is built for the combination.
inline int tex_id(int dtype, int mode, int degree)
{
    if (mode == kDispNone) return kTexNone;
    if (mode == kDispAlongRay) return dtype == 0 ? kTexF32Ray : dtype == 1 ? kTexF16Ray : kTexU8Ray;
    if (mode == kDispShVec3) {
        if (dtype == 0 && degree == 1) return kTexF32Vec3D1;
        if (dtype == 1 && degree == 2) return kTexF16Vec3D2;
        if (dtype == 2 && degree == 2) return kTexU8Vec3D2;
        if (degree < 0 || degree > 3) return -1;
        return dtype == 0 ? kTexF32Vec3 : dtype == 1 ? kTexF16Vec3 : kTexU8Vec3;
    }
    return -1;
}

// Eq. 2's vector form at any degree (0..3, taken at run time) for a dtype.
inline int tex_id_any_degree(int dtype)
{
    return dtype == 0 ? kTexF32Vec3 : dtype == 1 ? kTexF16Vec3 : kTexU8Vec3;
}

struct RenderLaunch {
    RayParams rp;
    GridParams gp;
    const _Float16 *weights;
    float4 *out;
    int view_sh;
    int tex;          // TexId
    bool tf16;
    int F, in, hid, nhid;
    int hid_w;        // hidden width of the weights (<= hid, the kernel's)
    int cus;
    int64_t l2_bytes;   // L2 of one XCD
    int blocks_mode;    // 0: by the gathers' line sharing, 1: all that fit, 2: two per CU
    int tile_stripe;    // > 0: stripe width of the tile order in tiles; <= 0: the default
    int chunk;          // > 0: early-termination path with this many samples per round
    int block_levels;   // finest levels with 16-byte block gathers: > 0 that many,
                        // < 0 none, 0 the default rule
    unsigned int *work; // device, kWorkWords words of work counters (zero)
};

bool render_variant_supported(int tex, int F, bool tf16, int in, int hid, int nhid);
bool mlp_variant_supported(int in, int hid, int nhid);

hipError_t launch_render(const RenderLaunch &L, hipStream_t stream);
// The phase-timer build's per-phase shader clocks (8 words, see
// mixrt_render.hip), after waiting for the device; hipErrorNotSupported in
// other builds.
hipError_t phase_cycles_read(uint64_t *out, bool reset);
// The grid size, tile-order stripe, samples per round, first level of
// 16-byte block gathers and hashed levels per batch of gathers launch_render
// would use (no launch).
hipError_t render_launch_shape(const RenderLaunch &L, int *blocks, int *stripe, int *chunk,
                               int *block_from, int *hash_batch, int *claims);
hipError_t launch_ray_setup(const RayParams &rp, int tex, float *out_x, int32_t *out_hit,
                            hipStream_t stream);
hipError_t launch_hash_encode(const GridParams &gp, int F, bool tf16, const float *x, int64_t n,
                              int32_t *oc, uint32_t *oi, float *ow, float *of, hipStream_t stream);
hipError_t launch_mlp(int in, int hid, int nhid, int hid_w, const _Float16 *weights,
                      const _Float16 *x, int64_t n, float4 *out4, int cus, hipStream_t stream);
hipError_t launch_composite(const float4 *srgb, int64_t rays, int K, float delta, float t_term,
                            const float *bg, float4 *out, hipStream_t stream);

}  // namespace mixrt
