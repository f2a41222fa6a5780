// The coarse-mesh hit per pixel (Fig. 2 step 1) by rasterisation, as the
// paper obtains it, on compute units: a visibility buffer of 64-bit keys
// (t bits << 32 | triangle) kept with atomic min, so the closest hit wins and
// equal t goes to the lower triangle index.  Coverage and depth come from the
// same fp32 ray-triangle test, on the same per-pixel rays, as the ray cast
// (mixrt_raycast.hip).
//
//   clear:   every pixel's key = all ones (no hit);
//   raster:  each wave takes 64 triangles of one view (strided over the
//            mesh, for balance between waves), clips them against a
//            plane just in front of the camera, projects them and bounds
//            their pixels (one pixel of margin); the (triangle, pixel) pairs
//            of all 64 boxes, in box order, are cut into 64 equal runs, one
//            per lane, so large and small triangles balance within the wave;
//            a lane finds its first box by binary search and then steps
//            pixel by pixel, box by box, testing with the pixel's ray
//            direction before normalisation (same order of hits);
//   resolve: per pixel, the winning triangle's hit is recomputed to write t,
//            the barycentric uv and the face normal.
// The winner of a pixel is the fp32 closest hit of its ray as the ray cast
// finds it, except where two triangles' hits lie within rounding of each
// other.  The keys live in the first 8 bytes of each 16-byte G-buffer record: the
// three launches need no memory beyond the caller's output.
#include "mixrt_common.hpp"
#include "mixrt_mesh.hpp"

namespace mixrt {

namespace {

constexpr uint64_t kNoHit = ~0ull;

__device__ __forceinline__ bool tri_hit(const float4 &A, const float4 &E1, const float4 &E2,
                                        const Ray &ray, float &t, float &b1, float &b2)
{
    const float px = ray.dy * E2.z - ray.dz * E2.y;
    const float py = ray.dz * E2.x - ray.dx * E2.z;
    const float pz = ray.dx * E2.y - ray.dy * E2.x;
    const float det = E1.x * px + E1.y * py + E1.z * pz;
    const float inv = __builtin_amdgcn_rcpf(det);
    const float sx = ray.ox - A.x, sy = ray.oy - A.y, sz = ray.oz - A.z;
    b1 = (sx * px + sy * py + sz * pz) * inv;
    const float qx = sy * E1.z - sz * E1.y;
    const float qy = sz * E1.x - sx * E1.z;
    const float qz = sx * E1.y - sy * E1.x;
    b2 = (ray.dx * qx + ray.dy * qy + ray.dz * qz) * inv;
    t = (E2.x * qx + E2.y * qy + E2.z * qz) * inv;
    return b1 >= 0.0f && b2 >= 0.0f && b1 + b2 <= 1.0f && t > MIXRT_RAY_T_MIN;
}

// The same test for a ray o + s D with D not normalised: s = t / |D|, so the
// order of hits along the ray is that of t, and t > t_min reads
// s^2 |D|^2 > t_min^2 (dd = |D|^2).  Returns s in `key_t`.
__device__ __forceinline__ bool tri_hit_scaled(const float4 &A, const float4 &E1, const float4 &E2,
                                               float ox, float oy, float oz, float dx, float dy,
                                               float dz, float dd, float &key_t)
{
    const float px = dy * E2.z - dz * E2.y;
    const float py = dz * E2.x - dx * E2.z;
    const float pz = dx * E2.y - dy * E2.x;
    const float det = E1.x * px + E1.y * py + E1.z * pz;
    const float inv = __builtin_amdgcn_rcpf(det);
    const float sx = ox - A.x, sy = oy - A.y, sz = oz - A.z;
    const float b1 = (sx * px + sy * py + sz * pz) * inv;
    const float qx = sy * E1.z - sz * E1.y;
    const float qy = sz * E1.x - sx * E1.z;
    const float qz = sx * E1.y - sy * E1.x;
    const float b2 = (dx * qx + dy * qy + dz * qz) * inv;
    const float s = (E2.x * qx + E2.y * qy + E2.z * qz) * inv;
    key_t = s;
    return b1 >= 0.0f && b2 >= 0.0f && b1 + b2 <= 1.0f && s > 0.0f &&
           s * s * dd > MIXRT_RAY_T_MIN * MIXRT_RAY_T_MIN;
}

__global__ __launch_bounds__(kBlock) void clear_kernel(uint4 *__restrict__ g0, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i < n) g0[i] = make_uint4(0xffffffffu, 0xffffffffu, 0u, 0u);
}

struct Box {
    float4 a, e1, e2;
    int x0, y0, bw, bh;
    uint32_t end;   // inclusive prefix sum of the wave's box areas
};

// Pixel box of a triangle in view c (empty: bw = bh = 0).
__device__ __forceinline__ void pixel_box(const RasterLaunch &L, const CamK &c, float zn,
                                          const float4 &A, const float4 &E1, const float4 &E2,
                                          int &x0, int &y0, int &bw, int &bh)
{
    // camera-space corners: R^T (p - o)
    float X[3], Y[3], Z[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const float wx = A.x + (k == 1 ? E1.x : (k == 2 ? E2.x : 0.0f)) - c.o[0];
        const float wy = A.y + (k == 1 ? E1.y : (k == 2 ? E2.y : 0.0f)) - c.o[1];
        const float wz = A.z + (k == 1 ? E1.z : (k == 2 ? E2.z : 0.0f)) - c.o[2];
        X[k] = c.R[0] * wx + c.R[3] * wy + c.R[6] * wz;
        Y[k] = c.R[1] * wx + c.R[4] * wy + c.R[7] * wz;
        Z[k] = c.R[2] * wx + c.R[5] * wy + c.R[8] * wz;
    }
    // clip against Z = -zn (the polygon in front has at most 4 corners) and
    // bound its projection; pixel i's centre is at W/2 + X/(-Z) f - ... (i + 0.5)
    const float f = 1.0f / c.inv_f;
    float lox = INFINITY, hix = -INFINITY, loy = INFINITY, hiy = -INFINITY;
    auto add = [&](float x, float y, float z) {
        const float s = f / (-z);
        const float sx = 0.5f * (float)L.W + x * s, sy = 0.5f * (float)L.H - y * s;
        lox = fminf(lox, sx);
        hix = fmaxf(hix, sx);
        loy = fminf(loy, sy);
        hiy = fmaxf(hiy, sy);
    };
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const int n = k == 2 ? 0 : k + 1;
        const bool in_k = Z[k] < -zn, in_n = Z[n] < -zn;
        if (in_k) add(X[k], Y[k], Z[k]);
        if (in_k != in_n) {
            const float s = (-zn - Z[k]) / (Z[n] - Z[k]);
            add(X[k] + s * (X[n] - X[k]), Y[k] + s * (Y[n] - Y[k]), -zn);
        }
    }
    x0 = y0 = bw = bh = 0;
    if (!(lox <= hix) || !(loy <= hiy)) return;   // nothing in front, or NaN
    // centres i + 0.5 in [lox, hix], one pixel of margin, clamped in float
    // before the conversion
    const float fx0 = fmaxf(floorf(lox - 0.5f) - 1.0f, 0.0f);
    const float fx1 = fminf(ceilf(hix - 0.5f) + 1.0f, (float)(L.W - 1));
    const float fy0 = fmaxf(floorf(loy - 0.5f) - 1.0f, 0.0f);
    const float fy1 = fminf(ceilf(hiy - 0.5f) + 1.0f, (float)(L.H - 1));
    if (!(fx0 <= fx1) || !(fy0 <= fy1)) return;
    x0 = (int)fx0;
    y0 = (int)fy0;
    bw = (int)fx1 - x0 + 1;
    bh = (int)fy1 - y0 + 1;
}

__global__ __launch_bounds__(kBlock) void raster_kernel(const RasterLaunch L)
{
    __shared__ Box s_box[kWavesPerBlock][kWave];
    const int view = blockIdx.y;
    const int wv = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
    // Triangles are dealt to waves with a stride of the wave count, so that
    // the large boxes of a nearby object (consecutive triangles) spread over
    // many waves instead of piling into a few.
    const int64_t n_waves = (int64_t)gridDim.x * kWavesPerBlock;
    const int64_t tri = (int64_t)lane * n_waves + (int64_t)blockIdx.x * kWavesPerBlock + wv;
    const CamK &c = L.cams[view];
    Box b;
    b.a = b.e1 = b.e2 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    b.x0 = b.y0 = b.bw = b.bh = 0;
    if (tri < L.n_faces) {
        b.a = L.tris[3 * tri];
        b.e1 = L.tris[3 * tri + 1];
        b.e2 = L.tris[3 * tri + 2];
        pixel_box(L, c, L.near_z[view], b.a, b.e1, b.e2, b.x0, b.y0, b.bw, b.bh);
    }
    // inclusive prefix sum of the box areas over the wave
    uint32_t end = (uint32_t)b.bw * (uint32_t)b.bh;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint32_t o = __shfl_up(end, d);
        if (lane >= d) end += o;
    }
    b.end = end;
    s_box[wv][lane] = b;
    const uint32_t total = __shfl(end, kWave - 1);
    wave_lds_sync();
    // this lane's run of pairs [q0, q1)
    const uint32_t q0 = (uint32_t)(((uint64_t)total * lane) >> 6);
    const uint32_t q1 = (uint32_t)(((uint64_t)total * (lane + 1)) >> 6);
    if (q0 >= q1) return;
    // first box whose end exceeds q0
    int cur = 0;
#pragma unroll
    for (int step = kWave / 2; step > 0; step >>= 1)
        if (s_box[wv][cur + step - 1].end <= q0) cur += step;
    const Box *bx = &s_box[wv][cur];
    uint32_t local = q0 - (cur ? s_box[wv][cur - 1].end : 0u);
    int j = (int)(local / (uint32_t)bx->bw);
    int i = (int)(local - (uint32_t)j * (uint32_t)bx->bw);
    float4 A = bx->a, E1 = bx->e1, E2 = bx->e2;
    int x0 = bx->x0, y0 = bx->y0, bw = bx->bw, bh = bx->bh;
    uint64_t *vis = (uint64_t *)L.g0;
    const int64_t view_base = (int64_t)view * L.H * L.W;
    for (uint32_t q = q0; q < q1; ++q) {
        const int px = x0 + i, py = y0 + j;
        // the pixel's ray direction before normalisation (as in camera_ray)
        const float cx = ((float)px + 0.5f - 0.5f * (float)L.W) * c.inv_f;
        const float cy = -(((float)py + 0.5f - 0.5f * (float)L.H) * c.inv_f);
        const float dx = c.R[0] * cx + c.R[1] * cy - c.R[2];
        const float dy = c.R[3] * cx + c.R[4] * cy - c.R[5];
        const float dz = c.R[6] * cx + c.R[7] * cy - c.R[8];
        float st;
        if (tri_hit_scaled(A, E1, E2, c.o[0], c.o[1], c.o[2], dx, dy, dz,
                           dx * dx + dy * dy + dz * dz, st)) {
            const uint64_t key = ((uint64_t)__float_as_uint(st) << 32) | (uint32_t)__float_as_int(A.w);
            atomicMin((unsigned long long *)&vis[2 * (view_base + (int64_t)py * L.W + px)],
                      (unsigned long long)key);
        }
        if (++i == bw) {
            i = 0;
            if (++j == bh && q + 1 < q1) {
                // next box with pixels (empty boxes hold no pair)
                do {
                    ++cur;
                } while (s_box[wv][cur].bw * s_box[wv][cur].bh == 0);
                bx = &s_box[wv][cur];
                A = bx->a;
                E1 = bx->e1;
                E2 = bx->e2;
                x0 = bx->x0;
                y0 = bx->y0;
                bw = bx->bw;
                bh = bx->bh;
                j = 0;
            }
        }
    }
}

__global__ __launch_bounds__(kBlock) void resolve_kernel(const RasterLaunch L)
{
    const int64_t pix = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t hw = (int64_t)L.H * L.W;
    if (pix >= (int64_t)L.views * hw) return;
    const uint64_t key = ((const uint64_t *)L.g0)[2 * pix];
    if (key == kNoHit) {
        L.g0[pix] = make_float4(-1.0f, 0.0f, 0.0f, 0.0f);
        if (L.g1) L.g1[pix] = make_float4(0.0f, 0.0f, 0.0f, __int_as_float(-1));
        return;
    }
    const int32_t id = (int32_t)(uint32_t)key;
    const int view = (int)(pix / hw);
    const int64_t rem = pix - (int64_t)view * hw;
    const int py = (int)(rem / L.W), px = (int)(rem - (int64_t)py * L.W);
    const Ray r = camera_ray(L.cams[view], L.W, L.H, (uint32_t)px, (uint32_t)py);
    const float4 A = L.tris[3 * (int64_t)id], E1 = L.tris[3 * (int64_t)id + 1],
                 E2 = L.tris[3 * (int64_t)id + 2];
    float t, b1, b2;
    tri_hit(A, E1, E2, r, t, b1, b2);   // the same arithmetic that won the pixel
    const float4 a0 = L.attr[2 * (int64_t)id], a1 = L.attr[2 * (int64_t)id + 1];
    const float b0 = 1.0f - b1 - b2;
    L.g0[pix] = make_float4(t, b0 * a0.x + b1 * a0.z + b2 * a1.x, b0 * a0.y + b1 * a0.w + b2 * a1.y,
                            0.0f);
    if (L.g1) {
        const float nx = E1.y * E2.z - E1.z * E2.y;
        const float ny = E1.z * E2.x - E1.x * E2.z;
        const float nz = E1.x * E2.y - E1.y * E2.x;
        const float nn = sqrtf(nx * nx + ny * ny + nz * nz);
        const float s = nn > 0.0f ? 1.0f / nn : 0.0f;
        L.g1[pix] = make_float4(nx * s, ny * s, nz * s, __int_as_float(id));
    }
}

}  // namespace

hipError_t launch_rasterize(const RasterLaunch &L, hipStream_t stream)
{
    const int64_t pixels = (int64_t)L.views * L.H * L.W;
    const int pix_blocks = (int)((pixels + kBlock - 1) / kBlock);
    hipLaunchKernelGGL(clear_kernel, dim3(pix_blocks), dim3(kBlock), 0, stream, (uint4 *)L.g0,
                       pixels);
    const int tri_blocks = (int)(((int64_t)L.n_faces + kBlock - 1) / kBlock);
    hipLaunchKernelGGL(raster_kernel, dim3(tri_blocks, L.views), dim3(kBlock), 0, stream, L);
    hipLaunchKernelGGL(resolve_kernel, dim3(pix_blocks), dim3(kBlock), 0, stream, L);
    return hipGetLastError();
}

}  // namespace mixrt
