// Internal interface between the C ABI (mixrt_api.cpp) and the kernels
// (mixrt_render.hip, mixrt_stages.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <type_traits>

#include "mixrt_device.hpp"

namespace mixrt {

struct RenderLaunch {
    RayParams rp;
    GridParams gp;
    const _Float16 *weights;
    float4 *out;
    int view_sh;
    bool xf16, tf16;
    int F, in, hid, nhid;
    int cus;
};

bool render_variant_supported(bool xf16, int F, bool tf16, int in, int hid, int nhid);
bool mlp_variant_supported(int in, int hid, int nhid);

hipError_t launch_render(const RenderLaunch &L, hipStream_t stream);
hipError_t launch_ray_setup(const RayParams &rp, bool xf16, float *out_x, int32_t *out_hit,
                            hipStream_t stream);
hipError_t launch_hash_encode(const GridParams &gp, int F, bool tf16, const float *x, int64_t n,
                              int32_t *oc, uint32_t *oi, float *ow, float *of, hipStream_t stream);
hipError_t launch_mlp(int in, int hid, int nhid, const _Float16 *weights, const _Float16 *x,
                      int64_t n, float4 *out4, int cus, hipStream_t stream);
hipError_t launch_composite(const float4 *srgb, int64_t rays, int K, float delta, float t_term,
                            const float *bg, float4 *out, hipStream_t stream);

}  // namespace mixrt
