// The coarse-mesh hit per pixel (Fig. 2 step 1) by ray casting: each lane
// takes one pixel's ray (the same fp32 ray the rendering kernel builds),
// walks the uniform grid's cells in the order the ray crosses them (3D DDA),
// intersects the triangles listed in each cell (Moller-Trumbore in fp32) and
// stops after the first cell whose exit distance is beyond the closest hit.
// Empty space is crossed in leaps: an empty cell at Chebyshev distance D from
// the nearest occupied cell sits in a cube of (2D-1)^3 empty cells, so the ray
// moves straight to the face where it leaves that cube.
//
// Launch shape: one 256-lane block per 16 x 16 pixel tile, each wave an 8 x 8
// quadrant, so the 64 rays of a wave cross nearly the same cells and their
// cell-list and triangle loads coalesce into few cache lines.  Neighbouring
// tiles are mapped to the same XCD so that its L2 holds the cells they share.
#include "mixrt_common.hpp"
#include "mixrt_mesh.hpp"

namespace mixrt {

namespace {

constexpr int kTile = 16;
constexpr float kInf = __builtin_inff();

struct Hit {
    float t, b1, b2;
    int32_t id;
    uint32_t ref;
};

struct Tri {
    float4 a, e1, e2;
};

__device__ __forceinline__ Tri load_tri(const float4 *__restrict__ refs, uint32_t r)
{
    return Tri{refs[3 * r], refs[3 * r + 1], refs[3 * r + 2]};
}

__device__ __forceinline__ void test_tri(const Tri &T, uint32_t r, const Ray &ray, Hit &h)
{
    const float4 &A = T.a, &E1 = T.e1, &E2 = T.e2;
    const float px = ray.dy * E2.z - ray.dz * E2.y;
    const float py = ray.dz * E2.x - ray.dx * E2.z;
    const float pz = ray.dx * E2.y - ray.dy * E2.x;
    const float det = E1.x * px + E1.y * py + E1.z * pz;
    // det = 0 (a ray in the triangle's plane) gives an infinite or NaN
    // barycentric below, which the comparisons reject.
    const float inv = __builtin_amdgcn_rcpf(det);
    const float sx = ray.ox - A.x, sy = ray.oy - A.y, sz = ray.oz - A.z;
    const float b1 = (sx * px + sy * py + sz * pz) * inv;
    const float qx = sy * E1.z - sz * E1.y;
    const float qy = sz * E1.x - sx * E1.z;
    const float qz = sx * E1.y - sy * E1.x;
    const float b2 = (ray.dx * qx + ray.dy * qy + ray.dz * qz) * inv;
    const float t = (E2.x * qx + E2.y * qy + E2.z * qz) * inv;
    const int32_t id = __float_as_int(A.w);
    if (b1 >= 0.0f && b2 >= 0.0f && b1 + b2 <= 1.0f && t > MIXRT_RAY_T_MIN &&
        (t < h.t || (t == h.t && id < h.id))) {
        h.t = t;
        h.b1 = b1;
        h.b2 = b2;
        h.id = id;
        h.ref = r;
    }
}

// Distance to the next cell face on one axis from cell c.
__device__ __forceinline__ float next_face(const MeshGridK &g, int a, int c, int step, float o,
                                           float inv)
{
    return (g.lo[a] + (float)(c + (step > 0)) * g.cell[a] - o) * inv;
}

// The walk's state: current cell, step direction and the distance to the
// next face on each axis.
struct Walk {
    int c[3], st[3];
    float tn[3];
};

// Move to the next cell: one DDA step (leap <= 1), or out of the empty cube
// c +- (leap - 1) through its nearest face, where that axis moves leap cells
// and the others go to the cell holding the exit point, kept inside the cube
// and never moved backwards.  False once the ray leaves the grid.
__device__ __forceinline__ bool advance(const MeshGridK &g, const float o[3], const float d[3],
                                        const float inv[3], int leap, Walk &w)
{
    if (leap <= 1) {
        const int ax = (w.tn[0] <= w.tn[1] && w.tn[0] <= w.tn[2]) ? 0 : (w.tn[1] <= w.tn[2] ? 1 : 2);
        int ca = 0;
#pragma unroll
        for (int a = 0; a < 3; ++a)
            if (a == ax) ca = w.c[a] + w.st[a];
        if (ca < 0 || ca >= g.n[ax]) return false;
#pragma unroll
        for (int a = 0; a < 3; ++a)
            if (a == ax) {
                w.c[a] = ca;
                w.tn[a] = next_face(g, a, ca, w.st[a], o[a], inv[a]);
            }
        return true;
    }
    float te[3];
#pragma unroll
    for (int a = 0; a < 3; ++a)
        te[a] = w.st[a] ? next_face(g, a, w.c[a] + w.st[a] * (leap - 1), w.st[a], o[a], inv[a]) : kInf;
    const int ax = (te[0] <= te[1] && te[0] <= te[2]) ? 0 : (te[1] <= te[2] ? 1 : 2);
    const float t = fminf(te[0], fminf(te[1], te[2]));
    bool out = false;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        int ca;
        if (a == ax) {
            ca = w.c[a] + w.st[a] * leap;
        } else if (w.st[a] == 0) {
            ca = w.c[a];
        } else {
            ca = (int)floorf((o[a] + t * d[a] - g.lo[a]) * g.inv_cell[a]);
            const int lo_a = w.st[a] > 0 ? w.c[a] : w.c[a] - (leap - 1);
            const int hi_a = w.st[a] < 0 ? w.c[a] : w.c[a] + (leap - 1);
            ca = min(max(ca, lo_a), hi_a);
        }
        out |= ca < 0 || ca >= g.n[a];
        w.c[a] = ca;
    }
    if (out) return false;
#pragma unroll
    for (int a = 0; a < 3; ++a)
        w.tn[a] = w.st[a] ? next_face(g, a, w.c[a], w.st[a], o[a], inv[a]) : kInf;
    return true;
}

__device__ __forceinline__ uint2 cell_rec(const MeshGridK &g, const Walk &w)
{
    return g.cells[((uint32_t)w.c[2] * (uint32_t)g.n[1] + (uint32_t)w.c[1]) * (uint32_t)g.n[0] +
                   (uint32_t)w.c[0]];
}

__device__ __forceinline__ Hit cast(const MeshGridK &g, const Ray &r)
{
    Hit h{kInf, 0.0f, 0.0f, INT32_MAX, 0u};
    const float o[3] = {r.ox, r.oy, r.oz}, d[3] = {r.dx, r.dy, r.dz};
    float inv[3], t0 = 0.0f, t1 = kInf;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        inv[a] = 1.0f / d[a];
        const float ta = (g.lo[a] - o[a]) * inv[a], tb = (g.hi[a] - o[a]) * inv[a];
        t0 = fmaxf(t0, fminf(ta, tb));
        t1 = fminf(t1, fmaxf(ta, tb));
    }
    if (!(t0 <= t1) || !(t0 < kInf)) return h;
    Walk w;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        const int ca = (int)floorf((o[a] + t0 * d[a] - g.lo[a]) * g.inv_cell[a]);
        w.c[a] = min(max(ca, 0), g.n[a] - 1);
        w.st[a] = d[a] > 0.0f ? 1 : (d[a] < 0.0f ? -1 : 0);
        w.tn[a] = w.st[a] ? next_face(g, a, w.c[a], w.st[a], o[a], inv[a]) : kInf;
    }
    // Every move goes at least one cell along the ray's direction on some
    // axis and never back on any, so the walk leaves the grid within
    // nx + ny + nz moves; the counter bounds it whatever the rounding.
    int steps = g.n[0] + g.n[1] + g.n[2];
    uint2 rec = cell_rec(g, w);
    for (;;) {
        // Traversal: every lane moves on until it stands in a cell with
        // triangles, so that the lanes of a wave test triangles together.
        bool alive = true;
        while (rec.y == 0) {
            if (--steps <= 0 || !advance(g, o, d, inv, (int)rec.x, w)) {
                alive = false;
                break;
            }
            rec = cell_rec(g, w);
        }
        if (!alive) break;
        // Intersection, with the next record's loads issued before the
        // current one is tested (the last index is reloaded, never passed).
        const uint32_t e = rec.x + rec.y;
        Tri T = load_tri(g.refs, rec.x);
        for (uint32_t k = rec.x; k < e; ++k) {
            const Tri nT = load_tri(g.refs, k + 1 < e ? k + 1 : k);
            test_tri(T, k, r, h);
            T = nT;
        }
        if (h.t <= fminf(w.tn[0], fminf(w.tn[1], w.tn[2]))) break;
        if (--steps <= 0 || !advance(g, o, d, inv, 1, w)) break;
        rec = cell_rec(g, w);
    }
    return h;
}

__global__ __launch_bounds__(kBlock) void raycast_kernel(const RaycastLaunch L)
{
    const int tiles_x = (L.W + kTile - 1) / kTile, tiles_y = (L.H + kTile - 1) / kTile;
    const int per_view = tiles_x * tiles_y;
    const int b = xcd_logical_block((int)blockIdx.x, (int)gridDim.x);
    const int view = b / per_view, rem = b - view * per_view;
    const int ty = rem / tiles_x, tx = rem - ty * tiles_x;
    const int w = (int)threadIdx.x >> 6, l = (int)threadIdx.x & 63;
    const int i = tx * kTile + (w & 1) * 8 + (l & 7);
    const int j = ty * kTile + (w >> 1) * 8 + (l >> 3);
    if (i >= L.W || j >= L.H) return;
    const Ray r = camera_ray(L.cams[view], L.W, L.H, (uint32_t)i, (uint32_t)j);
    const Hit h = cast(L.grid, r);
    const size_t pix = ((size_t)view * L.H + j) * L.W + i;
    if (h.id == INT32_MAX) {
        L.g0[pix] = make_float4(-1.0f, 0.0f, 0.0f, 0.0f);
        if (L.g1) L.g1[pix] = make_float4(0.0f, 0.0f, 0.0f, __int_as_float(-1));
        return;
    }
    const float4 a0 = L.grid.attr[2 * h.id], a1 = L.grid.attr[2 * h.id + 1];
    const float b0 = 1.0f - h.b1 - h.b2;
    L.g0[pix] = make_float4(h.t, b0 * a0.x + h.b1 * a0.z + h.b2 * a1.x,
                            b0 * a0.y + h.b1 * a0.w + h.b2 * a1.y, 0.0f);
    if (L.g1) {
        const float4 E1 = L.grid.refs[3 * h.ref + 1], E2 = L.grid.refs[3 * h.ref + 2];
        const float nx = E1.y * E2.z - E1.z * E2.y;
        const float ny = E1.z * E2.x - E1.x * E2.z;
        const float nz = E1.x * E2.y - E1.y * E2.x;
        const float nn = sqrtf(nx * nx + ny * ny + nz * nz);
        const float s = nn > 0.0f ? 1.0f / nn : 0.0f;
        L.g1[pix] = make_float4(nx * s, ny * s, nz * s, __int_as_float(h.id));
    }
}

}  // namespace

hipError_t launch_raycast(const RaycastLaunch &L, hipStream_t stream)
{
    const int tiles = ((L.W + kTile - 1) / kTile) * ((L.H + kTile - 1) / kTile) * L.views;
    hipLaunchKernelGGL(raycast_kernel, dim3(tiles), dim3(kBlock), 0, stream, L);
    return hipGetLastError();
}

}  // namespace mixrt
