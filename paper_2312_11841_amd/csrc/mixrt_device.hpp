// Device building blocks of the MixRT per-pixel path for gfx950 (CDNA4).
//
// Every stage of the path is one inline device function here; the fused
// render kernel and the per-stage kernels call the same functions, so the
// stage entry points exercise exactly the arithmetic mixrt_render runs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace mixrt {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
// Under-aligned integers for loads of two neighbouring table entries, split
// into 32-bit words with shifts.  (An under-aligned ext_vector_type typedef
// had its second element read back as the first by this compiler, and
// structs get split into single-dword loads.)
typedef uint64_t u64a4 __attribute__((aligned(4)));
typedef unsigned __int128 u128a8 __attribute__((aligned(8)));

__device__ __forceinline__ h2 word_h2(uint32_t w) { return __builtin_bit_cast(h2, w); }
__device__ __forceinline__ uint32_t h2_word(h2 v) { return __builtin_bit_cast(uint32_t, v); }

constexpr int kMaxViews = 16;
constexpr int kMaxLevels = 32;
constexpr int kWave = 64;

// Per-view camera constants, prepared on the host from mixrt_camera.
struct CamK {
    float R[9];      // rotation, row-major
    float o[3];      // centre
    float inv_f;     // 1 / focal length in pixels: f = (H/2) / tan(fov_y/2)
    float bg[3];
};

struct RayParams {
    const float4 *g0;
    int32_t views, W, H;
    int32_t rays;           // views * H * W (< 2^31)
    const void *tex;        // displacement coefficients [R][R][C]
    const void *tex_scale;  // Eq. 2 scale map [R][R] (SH_VEC3)
    int32_t tex_R, tex_V, tex_C;
    int32_t tex_degree;             // SH degree of Eq. 2's vector form
    float q_scale[2], q_offset[2];  // 8-bit dequantisation: coefficients, scale
    int32_t K;
    float delta;
    float t_term;
    CamK cams[kMaxViews];
};

struct GridParams {
    const void *table;
    uint32_t T_mask;        // T - 1
    uint32_t log2_T;
    int32_t L;
    uint32_t dense_mask;    // bit l: level l indexes its vertices densely
    int32_t n_dense;        // dense levels form the prefix 0..n_dense-1
    uint32_t N[kMaxLevels];
    float Nf[kMaxLevels];   // N as float, and N - 1 (exact: N <= 2^20), so
    float Ntop[kMaxLevels]; // that no lane converts them
    int32_t block_from;     // levels from here on load x-neighbour corner pairs
                            // as 16-byte blocks (4-byte entries; L: none)
    int32_t hash_batch;     // hashed levels per batch of gathers: 2, or 4
                            // (entries of 8 or more bytes)
};

// --------------------------------------------------------------------------
// Sec. 3.1: one ray through the centre of each pixel.
// --------------------------------------------------------------------------
struct Ray {
    float ox, oy, oz;
    float dx, dy, dz;
    int32_t view;
};

// The ray through the centre of pixel (i, j) of a W x H view (Sec. 3.1).
__device__ __forceinline__ Ray camera_ray(const CamK &c, int32_t W, int32_t H, uint32_t i,
                                          uint32_t j)
{
    const float cx = ((float)i + 0.5f - 0.5f * (float)W) * c.inv_f;
    const float cy = -(((float)j + 0.5f - 0.5f * (float)H) * c.inv_f);
    float dx = c.R[0] * cx + c.R[1] * cy - c.R[2];
    float dy = c.R[3] * cx + c.R[4] * cy - c.R[5];
    float dz = c.R[6] * cx + c.R[7] * cy - c.R[8];
    const float inv = 1.0f / sqrtf(dx * dx + dy * dy + dz * dz);
    Ray r;
    r.ox = c.o[0];
    r.oy = c.o[1];
    r.oz = c.o[2];
    r.dx = dx * inv;
    r.dy = dy * inv;
    r.dz = dz * inv;
    r.view = 0;
    return r;
}

__device__ __forceinline__ Ray pixel_ray(const RayParams &p, int32_t ray)
{
    const uint32_t hw = (uint32_t)p.H * (uint32_t)p.W;
    const uint32_t view = (uint32_t)ray / hw;
    const uint32_t rem = (uint32_t)ray - view * hw;
    const uint32_t j = rem / (uint32_t)p.W;
    const uint32_t i = rem - j * (uint32_t)p.W;
    Ray r = camera_ray(p.cams[view], p.W, p.H, i, j);
    r.view = (int32_t)view;
    return r;
}

// --------------------------------------------------------------------------
// Real spherical harmonics of a unit direction, degrees 0..3 (16 functions,
// ordered by degree then m = -l..l, orthonormal, no Condon-Shortley phase).
// Written as Cartesian polynomials; the constants are the normalisations
// sqrt((2l+1)/(4 pi) (l-|m|)!/(l+|m|)!) (times sqrt 2 for m != 0) folded into
// each polynomial.
// --------------------------------------------------------------------------
template <int NB>
__device__ __forceinline__ void sh_basis(float x, float y, float z, float *Y)
{
    static_assert(NB >= 1 && NB <= 16, "degree <= 3");
    Y[0] = 0.28209479177387814f;
    if (NB > 1) Y[1] = 0.48860251190291992f * y;
    if (NB > 2) Y[2] = 0.48860251190291992f * z;
    if (NB > 3) Y[3] = 0.48860251190291992f * x;
    const float xx = x * x, yy = y * y, zz = z * z;
    if (NB > 4) Y[4] = 1.0925484305920792f * x * y;
    if (NB > 5) Y[5] = 1.0925484305920792f * y * z;
    if (NB > 6) Y[6] = 0.31539156525252005f * (3.0f * zz - 1.0f);
    if (NB > 7) Y[7] = 1.0925484305920792f * x * z;
    if (NB > 8) Y[8] = 0.54627421529603959f * (xx - yy);
    if (NB > 9) Y[9] = 0.59004358992664352f * y * (3.0f * xx - yy);
    if (NB > 10) Y[10] = 2.8906114426405538f * x * y * z;
    if (NB > 11) Y[11] = 0.45704579946446572f * y * (5.0f * zz - 1.0f);
    if (NB > 12) Y[12] = 0.37317633259011540f * z * (5.0f * zz - 3.0f);
    if (NB > 13) Y[13] = 0.45704579946446572f * x * (5.0f * zz - 1.0f);
    if (NB > 14) Y[14] = 1.4453057213202769f * z * (xx - yy);
    if (NB > 15) Y[15] = 0.59004358992664352f * x * (xx - 3.0f * yy);
}

// --------------------------------------------------------------------------
// Eq. 2: the view-dependent displacement of the hit point.
//
// Texture kinds: element type (fp32, fp16 or 8-bit with an affine
// dequantisation) and displacement form.  A texel's channels are read in
// 16-byte chunks when texels are whole 16-byte lines, else element by
// element.  Bilinear filtering (texel centres at (i + 0.5)/R, clamp to edge)
// is done in fp32 on dequantised values.
// --------------------------------------------------------------------------
enum DispMode { kDispAlongRay = 0, kDispShVec3 = 1, kDispNone = 2 };

// DEG < 0: Eq. 2's vector form with the SH degree (0..3) taken at run time.
template <typename XT, int MODE, int DEG = 0>
struct TexKind {
    typedef XT T;
    static constexpr int mode = MODE;
    static constexpr int degree = DEG;
    static constexpr int nb = (DEG + 1) * (DEG + 1);
};

__device__ __forceinline__ float tex_elem(float e, float, float) { return e; }
__device__ __forceinline__ float tex_elem(_Float16 e, float, float) { return (float)e; }
__device__ __forceinline__ float tex_elem(uint8_t e, float qs, float qo)
{
    return qo + qs * (float)e;
}

struct Bilinear {
    int64_t t[4];   // element offsets of the 4 taps' texels (times C)
    float w[4];
};

__device__ __forceinline__ Bilinear bilinear_taps(int R, int C, float u, float v)
{
    float a = u * (float)R - 0.5f;
    float b = v * (float)R - 0.5f;
    // keep non-finite or far-out coordinates on the edge texels
    a = fminf(fmaxf(a, -1.0f), (float)R);
    b = fminf(fmaxf(b, -1.0f), (float)R);
    if (!(a == a)) a = 0.0f;
    if (!(b == b)) b = 0.0f;
    const float fa = floorf(a), fb = floorf(b);
    const float wa = a - fa, wb = b - fb;
    const int i0 = (int)fa, j0 = (int)fb;
    const int ia0 = min(max(i0, 0), R - 1), ia1 = min(max(i0 + 1, 0), R - 1);
    const int jb0 = min(max(j0, 0), R - 1), jb1 = min(max(j0 + 1, 0), R - 1);
    Bilinear B;
    B.t[0] = ((int64_t)jb0 * R + ia0) * C;
    B.t[1] = ((int64_t)jb0 * R + ia1) * C;
    B.t[2] = ((int64_t)jb1 * R + ia0) * C;
    B.t[3] = ((int64_t)jb1 * R + ia1) * C;
    B.w[0] = (1.0f - wa) * (1.0f - wb);
    B.w[1] = wa * (1.0f - wb);
    B.w[2] = (1.0f - wa) * wb;
    B.w[3] = wa * wb;
    return B;
}

// The 4 tap weights with an 8-bit map's dequantisation folded in: the
// weights sum to one, so sum_k w_k (qo + qs e_k) = qo + sum_k (w_k qs) e_k,
// and a filtered channel costs one conversion and one fma per tap instead of
// two fmas.  fp32 and fp16 maps are read as stored (base 0, weights as is).
template <typename XT>
struct TapWeights {
    float w[4];
    float base;
    __device__ __forceinline__ TapWeights(const Bilinear &B, float qs, float qo)
    {
        constexpr bool Q = std::is_same<XT, uint8_t>::value;
#pragma unroll
        for (int k = 0; k < 4; ++k) w[k] = Q ? B.w[k] * qs : B.w[k];
        base = Q ? qo : 0.0f;
    }
};

// Filtered channels [c0, c0 + EPV) of one 16-byte chunk of every texel.
template <typename XT>
__device__ __forceinline__ void bilinear_chunk(const XT *tex, const Bilinear &B,
                                               const TapWeights<XT> &tw, int c0, float *m)
{
    constexpr int EPV = 16 / (int)sizeof(XT);
#pragma unroll
    for (int e = 0; e < EPV; ++e) m[e] = tw.base;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        XT e[EPV];
        *(uint4 *)e = *(const uint4 *)(tex + B.t[k] + c0);
#pragma unroll
        for (int i = 0; i < EPV; ++i) m[i] += tw.w[k] * (float)e[i];
    }
}

template <typename XT>
__device__ __forceinline__ float bilinear_elem(const XT *tex, const Bilinear &B,
                                               const TapWeights<XT> &tw, int c)
{
    float m = tw.base;
#pragma unroll
    for (int k = 0; k < 4; ++k) m += tw.w[k] * (float)tex[B.t[k] + c];
    return m;
}

// Eq. 2 as printed for SH degree DEG: S_a = sum_v Y_v(d) m[a nb + v] over
// nb = (DEG + 1)^2 harmonics per axis, and the offset m_s(p_t) S.
template <typename XT, int DEG>
__device__ __forceinline__ void vec3_offset(const RayParams &p, const Bilinear &B, float u,
                                            float v, const float *Y, bool vec, float &ox,
                                            float &oy, float &oz)
{
    constexpr int EPV = 16 / (int)sizeof(XT);
    constexpr int NB = (DEG + 1) * (DEG + 1), NCH = 3 * NB;
    constexpr int NCHUNK = (NCH + EPV - 1) / EPV;
    const XT *tex = (const XT *)p.tex;
    const TapWeights<XT> tw(B, p.q_scale[0], p.q_offset[0]);
    float m[NCHUNK * EPV];
    if (vec) {
#pragma unroll
        for (int q = 0; q < NCHUNK; ++q) bilinear_chunk<XT>(tex, B, tw, q * EPV, m + q * EPV);
    } else {
#pragma unroll
        for (int c = 0; c < NCH; ++c) m[c] = bilinear_elem<XT>(tex, B, tw, c);
    }
    const Bilinear Bs = bilinear_taps(p.tex_R, 1, u, v);
    const float ms = bilinear_elem<XT>((const XT *)p.tex_scale, Bs,
                                       TapWeights<XT>(Bs, p.q_scale[1], p.q_offset[1]), 0);
    float S[3] = {0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int vv = 0; vv < NB; ++vv) S[a] += Y[vv] * m[a * NB + vv];
    ox = ms * S[0];
    oy = ms * S[1];
    oz = ms * S[2];
}

// Offset p_cali - p for the ray direction d at texture coordinate (u, v).
template <typename TK>
__device__ __forceinline__ void displacement(const RayParams &p, float u, float v, float dx,
                                             float dy, float dz, float &ox, float &oy, float &oz)
{
    typedef typename TK::T XT;
    ox = oy = oz = 0.0f;
    if (TK::mode == kDispNone) return;
    constexpr int EPV = 16 / (int)sizeof(XT);
    const XT *tex = (const XT *)p.tex;
    const Bilinear B = bilinear_taps(p.tex_R, p.tex_C, u, v);
    const bool vec = ((p.tex_C * (int)sizeof(XT)) & 15) == 0;
    float Y[16];
    sh_basis<16>(dx, dy, dz, Y);
    if (TK::mode == kDispAlongRay) {
        // s = sum_v Y_v(d) m_v over the first V channels; p_cali = p + s d
        const TapWeights<XT> tw(B, p.q_scale[0], p.q_offset[0]);
        float s = 0.0f;
        if (vec) {
#pragma unroll
            for (int c0 = 0; c0 < 16; c0 += EPV) {
                if (c0 < p.tex_V) {
                    float m[EPV];
                    bilinear_chunk<XT>(tex, B, tw, c0, m);
#pragma unroll
                    for (int e = 0; e < EPV && c0 + e < 16; ++e)
                        if (c0 + e < p.tex_V) s += Y[c0 + e] * m[e];
                }
            }
        } else {
#pragma unroll
            for (int c = 0; c < 16; ++c)
                if (c < p.tex_V) s += Y[c] * bilinear_elem<XT>(tex, B, tw, c);
        }
        ox = s * dx;
        oy = s * dy;
        oz = s * dz;
    } else if (TK::degree >= 0) {
        vec3_offset<XT, (TK::degree >= 0 ? TK::degree : 0)>(p, B, u, v, Y, vec, ox, oy, oz);
    } else {
        switch (p.tex_degree) {
        case 0: vec3_offset<XT, 0>(p, B, u, v, Y, vec, ox, oy, oz); break;
        case 1: vec3_offset<XT, 1>(p, B, u, v, Y, vec, ox, oy, oz); break;
        case 2: vec3_offset<XT, 2>(p, B, u, v, Y, vec, ox, oy, oz); break;
        default: vec3_offset<XT, 3>(p, B, u, v, Y, vec, ox, oy, oz); break;
        }
    }
}

// --------------------------------------------------------------------------
// Sec. 2.1: contraction of unbounded space into the ball of radius 2
// (identity inside the unit ball, (2 - 1/r) q/r outside), then the affine
// map of [-2, 2]^3 onto the grid's unit cube.
// --------------------------------------------------------------------------
__device__ __forceinline__ void contract_to_cube(float qx, float qy, float qz, float &x0,
                                                 float &x1, float &x2)
{
    const float r2 = qx * qx + qy * qy + qz * qz;
    float s = 1.0f;
    if (r2 > 1.0f) {
        const float r = sqrtf(r2);
        s = (2.0f - 1.0f / r) / r;
    }
    x0 = fminf(fmaxf((qx * s + 2.0f) * 0.25f, 0.0f), 1.0f);
    x1 = fminf(fmaxf((qy * s + 2.0f) * 0.25f, 0.0f), 1.0f);
    x2 = fminf(fmaxf((qz * s + 2.0f) * 0.25f, 0.0f), 1.0f);
    if (!(x0 == x0)) x0 = 0.0f;
    if (!(x1 == x1)) x1 = 0.0f;
    if (!(x2 == x2)) x2 = 0.0f;
}

// The along-ray displacement computed jointly by the 8 lanes that hold
// samples of one ray (consecutive lanes, 8-aligned, all taking this call),
// when a texel is one 16-byte line: lane j loads half (j >> 2) of tap (j & 3),
// weighs its channels by the tap weight and the SH values, and three
// butterfly exchanges within the 8 lanes sum the partial products.  One
// 8-byte load per lane instead of four 16-byte loads.
template <typename TK>
__device__ __forceinline__ void displacement_ray8(const RayParams &p, float u, float v, float dx,
                                                  float dy, float dz, int sub, float &ox,
                                                  float &oy, float &oz)
{
    typedef typename TK::T XT;
    constexpr int EH = 8 / (int)sizeof(XT);   // channels in half a texel
    const XT *tex = (const XT *)p.tex;
    const Bilinear B = bilinear_taps(p.tex_R, p.tex_C, u, v);
    const int tap = sub & 3, half = (sub >> 2) & 1;
    int64_t off = B.t[0];
    float w = B.w[0];
#pragma unroll
    for (int q = 1; q < 4; ++q)
        if (tap == q) {
            off = B.t[q];
            w = B.w[q];
        }
    XT e[EH];
    *(uint2 *)e = *(const uint2 *)(tex + off + half * EH);
    float Y[16];
    sh_basis<16>(dx, dy, dz, Y);
    const float qs = p.q_scale[0], qo = p.q_offset[0];
    // the lane's SH values, picked by a bit mask (a select of two array
    // elements would become a dynamic index into a private array)
    const uint32_t pick = 0u - (uint32_t)half;
    float part = 0.0f;
#pragma unroll
    for (int i = 0; i < EH; ++i) {
        const float y = __uint_as_float((__float_as_uint(Y[i]) & ~pick) |
                                        (__float_as_uint(Y[EH + i]) & pick));
        if (half * EH + i < p.tex_V) part += y * tex_elem(e[i], qs, qo);
    }
    part *= w;
    part += __shfl_xor(part, 1);
    part += __shfl_xor(part, 2);
    part += __shfl_xor(part, 4);
    ox = part * dx;
    oy = part * dy;
    oz = part * dz;
}

// Whether displacement_ray8 serves a call: the along-ray form, 16-byte
// texels, and K a multiple of 8 dividing 64 (a ray's samples then sit in
// whole 8-lane groups).
template <typename TK>
__device__ __forceinline__ bool ray8_applies(const RayParams &p)
{
    return TK::mode == kDispAlongRay && p.tex_C * (int)sizeof(typename TK::T) == 16 &&
           (p.K & 7) == 0 && 64 % p.K == 0;
}

// A hit ray's calibrated frame: P = o + (p_cali - p), so that sample k sits
// at P + (t + (k - (K-1)/2) delta) d.
struct RayHit {
    float px, py, pz;
    float t;
};

// Hit test and Eq. 2 calibration of a ray (sub: the lane's index within its
// ray's 8-lane group when displacement_ray8 serves the call).  Returns false
// for a miss.
template <typename TK>
__device__ __forceinline__ bool ray_hit(const RayParams &p, const Ray &r, float4 g, int sub,
                                        RayHit &h)
{
    h.t = g.x;
    const bool hit = h.t > 0.0f && h.t < INFINITY;
    if (!hit) {
        h.px = h.py = h.pz = 0.0f;
        return false;
    }
    float ox, oy, oz;
    if (ray8_applies<TK>(p))
        displacement_ray8<TK>(p, g.y, g.z, r.dx, r.dy, r.dz, sub & 7, ox, oy, oz);
    else
        displacement<TK>(p, g.y, g.z, r.dx, r.dy, r.dz, ox, oy, oz);
    h.px = r.ox + ox;
    h.py = r.oy + oy;
    h.pz = r.oz + oz;
    return true;
}

// Sample k of a hit ray: placement along d, contraction, cube map.
__device__ __forceinline__ void sample_at(const RayParams &p, const RayHit &h, float dx, float dy,
                                          float dz, int k, float &x0, float &x1, float &x2)
{
    const float off = h.t + ((float)k - 0.5f * (float)(p.K - 1)) * p.delta;
    contract_to_cube(h.px + off * dx, h.py + off * dy, h.pz + off * dz, x0, x1, x2);
}

// Steps before the grid for sample k of a ray: hit test, Eq. 2 calibration,
// sample placement, contraction.  Returns false for a miss.
template <typename TK>
__device__ __forceinline__ bool sample_position(const RayParams &p, const Ray &r, float4 g, int k,
                                                float &x0, float &x1, float &x2)
{
    RayHit h;
    if (!ray_hit<TK>(p, r, g, k, h)) {
        x0 = x1 = x2 = 0.0f;
        return false;
    }
    sample_at(p, h, r.dx, r.dy, r.dz, k, x0, x1, x2);
    return true;
}

// --------------------------------------------------------------------------
// Sec. 3.1 / 4.3.3: one level of the multiresolution hash encoding.
// The voxel is chosen from the fp32 product x * N_l (one rounding, no
// contraction into an FMA) so corners and indices are reproducible.
// --------------------------------------------------------------------------
// Table reads use a uniform (scalar) level base plus a 32-bit byte offset,
// which maps onto the scalar-base + vector-offset form of global loads.
template <int F, bool F16>
struct TableEntry;

template <>
struct TableEntry<2, true> {
    static constexpr uint32_t kBytes = 4;
    static __device__ __forceinline__ void from_word(uint32_t w, float *v)
    {
        const h2 h = __builtin_bit_cast(h2, w);
        v[0] = (float)h.x;
        v[1] = (float)h.y;
    }
    static __device__ __forceinline__ void load(const char *t, uint32_t off, float *v)
    {
        from_word(*(const uint32_t *)(t + off), v);
    }
};

template <>
struct TableEntry<2, false> {
    static constexpr uint32_t kBytes = 8;
    static __device__ __forceinline__ void load(const char *t, uint32_t off, float *v)
    {
        const float2 f = *(const float2 *)(t + off);
        v[0] = f.x;
        v[1] = f.y;
    }
};

template <>
struct TableEntry<4, true> {
    static constexpr uint32_t kBytes = 8;
    static __device__ __forceinline__ void from_pair(const uint2 raw, float *v)
    {
        const h2 a = __builtin_bit_cast(h2, raw.x), b = __builtin_bit_cast(h2, raw.y);
        v[0] = (float)a.x;
        v[1] = (float)a.y;
        v[2] = (float)b.x;
        v[3] = (float)b.y;
    }
    static __device__ __forceinline__ void load(const char *t, uint32_t off, float *v)
    {
        const uint2 raw = *(const uint2 *)(t + off);
        const h2 a = __builtin_bit_cast(h2, raw.x), b = __builtin_bit_cast(h2, raw.y);
        v[0] = (float)a.x;
        v[1] = (float)a.y;
        v[2] = (float)b.x;
        v[3] = (float)b.y;
    }
};

template <>
struct TableEntry<4, false> {
    static constexpr uint32_t kBytes = 16;
    static __device__ __forceinline__ void load(const char *t, uint32_t off, float *v)
    {
        const float4 f = *(const float4 *)(t + off);
        v[0] = f.x;
        v[1] = f.y;
        v[2] = f.z;
        v[3] = f.w;
    }
};

// Two neighbouring entries (idx, idx + 1) in one load: along x, the dense
// index of corner (c0 + 1) is the dense index of c0 plus one.  Entries are
// at least 4-byte aligned, which multi-dword global loads accept.
template <int F, bool F16>
struct TablePair;

template <>
struct TablePair<2, true> {
    static __device__ __forceinline__ void load(const char *t, uint32_t off, float *v0, float *v1)
    {
        const uint64_t raw = *(const u64a4 *)(t + off);
        const h2 a = word_h2((uint32_t)raw), b = word_h2((uint32_t)(raw >> 32));
        v0[0] = (float)a.x;
        v0[1] = (float)a.y;
        v1[0] = (float)b.x;
        v1[1] = (float)b.y;
    }
};

template <>
struct TablePair<2, false> {
    static __device__ __forceinline__ void load(const char *t, uint32_t off, float *v0, float *v1)
    {
        const unsigned __int128 raw = *(const u128a8 *)(t + off);
        v0[0] = __builtin_bit_cast(float, (uint32_t)raw);
        v0[1] = __builtin_bit_cast(float, (uint32_t)(raw >> 32));
        v1[0] = __builtin_bit_cast(float, (uint32_t)(raw >> 64));
        v1[1] = __builtin_bit_cast(float, (uint32_t)(raw >> 96));
    }
};

template <>
struct TablePair<4, true> {
    static __device__ __forceinline__ void load(const char *t, uint32_t off, float *v0, float *v1)
    {
        const unsigned __int128 raw = *(const u128a8 *)(t + off);
        const h2 a = word_h2((uint32_t)raw), b = word_h2((uint32_t)(raw >> 32));
        const h2 c = word_h2((uint32_t)(raw >> 64)), d = word_h2((uint32_t)(raw >> 96));
        v0[0] = (float)a.x;
        v0[1] = (float)a.y;
        v0[2] = (float)b.x;
        v0[3] = (float)b.y;
        v1[0] = (float)c.x;
        v1[1] = (float)c.y;
        v1[2] = (float)d.x;
        v1[3] = (float)d.y;
    }
};

template <>
struct TablePair<4, false> {
    static __device__ __forceinline__ void load(const char *t, uint32_t off, float *v0, float *v1)
    {
        TableEntry<4, false>::load(t, off, v0);
        TableEntry<4, false>::load(t, off + 16u, v1);
    }
};

constexpr uint32_t kPrimeY = 2654435761u;
constexpr uint32_t kPrimeZ = 805459861u;

// Voxel, fractional position and the 8 corner entries of one query at one
// level, as byte offsets into the level's table for entries of EB bytes.
// Corner b has offset (b & 1, b >> 1 & 1, b >> 2 & 1).
struct LevelSetup {
    float cf[3];       // voxel corner c0 (integral values)
    float fr[3];
    uint32_t off[8];   // entry index times EB
};

// IN_UNIT: the query is known to lie in [0, 1]^3 (the render path clamps it
// there), so only the upper clamp of the voxel is needed.  Otherwise a
// coordinate below 0 or NaN takes voxel 0, as the oracle does.
//
// The byte offsets are computed directly: shifting left distributes over
// XOR and AND, so (h & (T - 1)) EB for a hash h = x ^ y pY ^ z pZ (mod 2^32)
// equals (x EB ^ y (pY EB) ^ z (pZ EB)) & ((T - 1) EB) with the products
// taken mod 2^32 (T EB <= 2^30), and a dense index scales term by term.
template <uint32_t EB, bool IN_UNIT>
__device__ __forceinline__ void level_setup(const GridParams &gp, int l, bool dense, float x0,
                                            float x1, float x2, LevelSetup &s)
{
    static_assert(EB == 4 || EB == 8 || EB == 16, "entry size");
    const uint32_t N = gp.N[l], T_mask = gp.T_mask;
    const float Nf = gp.Nf[l], top = gp.Ntop[l];
    // p = x N rounded once to fp32, as the oracle takes it.  The empty asm
    // keeps the compiler from fusing the product into p - c0 (which would
    // skip that rounding); with it, p - c0 is exact (c0 <= p < c0 + 1), so the
    // fractions equal the oracle's.
    float p[3] = {x0 * Nf, x1 * Nf, x2 * Nf};
#pragma unroll
    for (int a = 0; a < 3; ++a)
        asm("" : "+v"(p[a]));
    uint32_t c[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        if (IN_UNIT) {
            // 0 <= p <= N: truncation is the floor, clamped to N - 1 in
            // integers (the float clamp would first have to quiet p)
            c[a] = min((uint32_t)p[a], N - 1u);
            s.cf[a] = (float)c[a];
        } else {
            // floor(min(p, N - 1)) = min(floor(p), N - 1), N - 1 integral
            s.cf[a] = floorf(fminf(fmaxf(p[a], 0.0f), top));
            c[a] = (uint32_t)s.cf[a];
        }
        s.fr[a] = p[a] - s.cf[a];
    }
    if (dense) {
        const uint32_t s1 = N + 1u, s2 = s1 * s1;
        const uint32_t base = c[0] * EB + c[1] * (s1 * EB) + c[2] * (s2 * EB);
#pragma unroll
        for (int b = 0; b < 8; ++b)
            s.off[b] = base + ((b & 1) ? EB : 0u) + ((b & 2) ? s1 * EB : 0u) +
                       ((b & 4) ? s2 * EB : 0u);
    } else {
        constexpr uint32_t pY = kPrimeY * EB, pZ = kPrimeZ * EB;   // mod 2^32
        const uint32_t mask = T_mask * EB;
        const uint32_t hx0 = c[0] * EB, hx1 = hx0 + EB;
        const uint32_t hy0 = c[1] * pY, hy1 = hy0 + pY;
        const uint32_t hz0 = c[2] * pZ, hz1 = hz0 + pZ;
#pragma unroll
        for (int b = 0; b < 8; ++b)
            s.off[b] = (((b & 1) ? hx1 : hx0) ^ ((b & 2) ? hy1 : hy0) ^ ((b & 4) ? hz1 : hz0)) &
                       mask;
    }
}

__device__ __forceinline__ float corner_weight(const LevelSetup &s, int b)
{
    const float w0 = (b & 1) ? s.fr[0] : 1.0f - s.fr[0];
    const float w1 = (b & 2) ? s.fr[1] : 1.0f - s.fr[1];
    const float w2 = (b & 4) ? s.fr[2] : 1.0f - s.fr[2];
    return w0 * w1 * w2;
}

// Word i of an aligned 16-byte block, i = bits 2-3 of the entry's byte
// offset, picked with bit masks (as selects, the compiler turns the pick
// into an indexed read of a private copy of the block).  The empty asm
// statement hides that the masks are all zeros or all ones, so they stay
// one bitfield extract each and the picks three bitfield inserts, instead
// of compares into lane masks and selects that need wait states between
// them (block-gather frames 0.3-1% faster).
__device__ __forceinline__ uint32_t block_word(const uint4 &q, uint32_t off)
{
    uint32_t m8 = (uint32_t)__builtin_amdgcn_sbfe((int)off, 3, 1);   // bit 3 set: all ones
    uint32_t m4 = (uint32_t)__builtin_amdgcn_sbfe((int)off, 2, 1);   // bit 2 set: all ones
    asm volatile("" : "+v"(m8), "+v"(m4));
    const uint32_t lo = (q.z & m8) | (q.x & ~m8);
    const uint32_t hi = (q.w & m8) | (q.y & ~m8);
    return (hi & m4) | (lo & ~m4);
}

// Whether a hashed level's x-neighbour corners (2q, 2q + 1) can share one
// aligned 16-byte block: 4-byte entries only.  The hash multiplies x by one,
// so the entries of x and x + 1 differ in the index bits that x and x + 1
// differ in: bits 0-1 (the same block) unless x = 3 (mod 4).
template <int F, bool F16>
constexpr bool kBlockPairs = TableEntry<F, F16>::kBytes == 4;

// The same for 8-byte entries (F = 4 fp16, the deployed grid's): the
// entries of x and x + 1 share an aligned 16-byte block when x is even.
template <int F, bool F16>
constexpr bool kBlockPairs8 = F16 && TableEntry<F, F16>::kBytes == 8;

// The 8 corner entries of a level: 4 pair loads on a dense level, 8 single
// loads on a hashed one.  BLOCKS (hashed levels of 4- or 8-byte entries):
// one 16-byte block load per x-neighbour pair, which holds both entries in
// 3 voxels of 4 (4-byte entries) or 1 of 2 (8-byte entries), plus a load of
// each x + 1 entry in the lanes whose voxel straddles two blocks: 4 full
// gathers and 4 partial ones instead of 8 full ones.  The vector L1 charges
// a scattered gather by the lanes and distinct lines it touches whatever
// its width, so this pays on levels whose lanes touch distinct lines (the
// finest); where lanes share lines a 16-byte gather costs more than a
// narrower one and the word picks cost ALU work.
template <int F, bool F16, bool DENSE, bool BLOCKS = false>
__device__ __forceinline__ void level_fetch(const void *table_l, const LevelSetup &s,
                                            float (*v)[F])
{
    const char *t = (const char *)table_l;
    if constexpr (DENSE) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            TablePair<F, F16>::load(t, s.off[2 * q], v[2 * q], v[2 * q + 1]);
    } else if constexpr (BLOCKS && kBlockPairs<F, F16>) {
        // the pairs' offsets differ by the same x part (the y and z parts
        // cancel), so one test serves all four
        const bool straddle = (s.off[0] ^ s.off[1]) >= 16u;
        uint4 blk[4];
        uint32_t far[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int q = 0; q < 4; ++q)
            blk[q] = *(const uint4 *)(t + (s.off[2 * q] & ~15u));
        if (straddle) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                far[q] = *(const uint32_t *)(t + s.off[2 * q + 1]);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t w0 = block_word(blk[q], s.off[2 * q]);
            const uint32_t w1 = straddle ? far[q] : block_word(blk[q], s.off[2 * q + 1]);
            TableEntry<F, F16>::from_word(w0, v[2 * q]);
            TableEntry<F, F16>::from_word(w1, v[2 * q + 1]);
        }
    } else if constexpr (BLOCKS && kBlockPairs8<F, F16>) {
        // the entries of x and x + 1 differ in bit 0 of the index when x is
        // even (one block, the halves picked by bit 3 of the offset) and in
        // higher bits when x is odd (a straddle, the same for all four)
        const bool straddle = (s.off[0] ^ s.off[1]) >= 16u;
        uint4 blk[4];
        uint2 far[4] = {{0u, 0u}, {0u, 0u}, {0u, 0u}, {0u, 0u}};
#pragma unroll
        for (int q = 0; q < 4; ++q)
            blk[q] = *(const uint4 *)(t + (s.off[2 * q] & ~15u));
        if (straddle) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                far[q] = *(const uint2 *)(t + s.off[2 * q + 1]);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            // bit 3 set: the x entry is the block's upper half (a mask kept
            // opaque, as in block_word)
            uint32_t m = (uint32_t)__builtin_amdgcn_sbfe((int)s.off[2 * q], 3, 1);
            asm volatile("" : "+v"(m));
            const uint2 e0 = {(blk[q].z & m) | (blk[q].x & ~m), (blk[q].w & m) | (blk[q].y & ~m)};
            const uint2 e1o = {(blk[q].x & m) | (blk[q].z & ~m), (blk[q].y & m) | (blk[q].w & ~m)};
            const uint2 e1 = straddle ? far[q] : e1o;
            TableEntry<F, F16>::from_pair(e0, v[2 * q]);
            TableEntry<F, F16>::from_pair(e1, v[2 * q + 1]);
        }
    } else {
#pragma unroll
        for (int b = 0; b < 8; ++b)
            TableEntry<F, F16>::load(t, s.off[b], v[b]);
    }
}

template <int F>
__device__ __forceinline__ void level_accumulate(const LevelSetup &s, const float (*v)[F],
                                                 float *feat)
{
#pragma unroll
    for (int f = 0; f < F; ++f)
        feat[f] = 0.0f;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        const float w = corner_weight(s, b);
#pragma unroll
        for (int f = 0; f < F; ++f)
            feat[f] += w * v[b][f];
    }
}

__device__ __forceinline__ const void *level_base(const GridParams &g, int l, int F, bool f16)
{
    const size_t esz = f16 ? 2 : 4;
    return (const char *)g.table + (size_t)l * ((size_t)g.T_mask + 1) * (size_t)F * esz;
}

// G consecutive levels starting at l0, all of one kind (dense or hashed):
// every corner load of the group is issued before any interpolation, so a
// wave keeps 4G (dense) or 8G (hashed) gathers in flight.
template <int F, bool F16, int G, bool DENSE, bool BLOCKS = false>
__device__ __forceinline__ void hash_group(const GridParams &gp, int l0, float x0, float x1,
                                           float x2, float (*feat)[F])
{
    LevelSetup s[G];
    float v[G][8][F];
#pragma unroll
    for (int g = 0; g < G; ++g)
        level_setup<TableEntry<F, F16>::kBytes, true>(gp, l0 + g, DENSE, x0, x1, x2, s[g]);
#pragma unroll
    for (int g = 0; g < G; ++g)
        level_fetch<F, F16, DENSE, BLOCKS>(level_base(gp, l0 + g, F, F16), s[g], v[g]);
#pragma unroll
    for (int g = 0; g < G; ++g)
        level_accumulate<F>(s[g], v[g], feat[g]);
}

// --------------------------------------------------------------------------
// Sec. 3.1: the small MLP on MFMA.  One call evaluates 16 samples (one
// 16-wide N tile) of a wave: the layers are computed transposed,
// Z^T[out][sample] = W^T[out][in] X^T[in][sample], so the fp32 accumulator
// of one layer, after ReLU and conversion, is already the B operand of the
// next layer in registers (the input neurons are permuted consistently in
// the A operand instead of moving data across lanes).
//
// gfx950 lane layouts (wave64), lane l, c = l & 15, g = l >> 4:
//   mfma_f32_16x16x32_f16  A: row c, k = 8g..8g+7;  B: column c, k = 8g..8g+7
//   mfma_f32_16x16x16_f16  A: row c, k = 4g..4g+3;  B: column c, k = 4g..4g+3
//   D (both):              column c, rows 4g..4g+3
//
// The 32-deep K chunks of a tile accumulate in place (16x16x32 into
// 16x16x32, the same registers as C and D).  A 16-deep remainder starts from
// a zero accumulator and is added on the VALU: with this compiler, chains that
// fed a 16x16x32 result into a 16x16x16 accumulate (with a different
// destination register) read a stale accumulator on gfx950, while in-place
// 16x16x32 chains and zero-C products were exact.
// --------------------------------------------------------------------------

// Input slot -> neuron for a layer fed from the previous layer's registers.
// 32-wide chunk ch, slot 8g + j: tile 2ch + (j >> 2), row 4g + (j & 3).
__device__ __forceinline__ int perm32(int ch, int g, int j)
{
    return (2 * ch + (j >> 2)) * 16 + 4 * g + (j & 3);
}

template <int KIN, int MOUT, bool FROM_REGS>
struct LayerA {
    static constexpr int NC = KIN / 32;            // 32-deep chunks
    static constexpr int R16 = (KIN % 32) / 16;    // one trailing 16-deep chunk
    static constexpr int MT = (MOUT + 15) / 16;    // 16-row output tiles
    static_assert(KIN % 16 == 0, "input width must be a multiple of 16");
    static_assert(!FROM_REGS || KIN == 16 || KIN % 32 == 0, "hidden width 16, 32 or 64");
    h8 a32[MT][NC > 0 ? NC : 1];
    h4 a16[MT];

    // W: fp16 [kin][mout] row-major in global memory, a layer of logical
    // widths kin <= KIN, mout <= MOUT; the tile's other rows and columns are
    // zero, so a narrower layer (Tab. 3's 8 hidden neurons on the 16-wide
    // tile) is computed exactly: its padded neurons stay 0 through ReLU and
    // add nothing downstream.
    __device__ __forceinline__ void load(const _Float16 *W, int lane, int kin, int mout)
    {
        const int c = lane & 15, g = lane >> 4;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int o = mt * 16 + c;
            const bool ok = o < mout;
#pragma unroll
            for (int ch = 0; ch < NC; ++ch) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int k = FROM_REGS ? perm32(ch, g, j) : ch * 32 + 8 * g + j;
                    a32[mt][ch][j] = ok && k < kin ? W[k * mout + o] : (_Float16)0.0f;
                }
            }
            if (R16) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int k = NC * 32 + 4 * g + j;
                    a16[mt][j] = ok && k < kin ? W[k * mout + o] : (_Float16)0.0f;
                }
            }
        }
    }
};

// Activations of one 16-sample tile held as MFMA D fragments: acc[t][j] is
// neuron 16t + 4g + j of sample column c.
template <int W>
struct Act {
    static constexpr int MT = (W + 15) / 16;
    f4 acc[MT];
};

// ReLU of two fp32 activations, packed to fp16 (max commutes with rounding).
__device__ __forceinline__ h2 relu_pack(float a, float b)
{
    const h2 v = {(_Float16)a, (_Float16)b};
    const h2 z = {(_Float16)0.0f, (_Float16)0.0f};
    return __builtin_elementwise_max(v, z);
}

template <int NC, int R16, typename AL>
__device__ __forceinline__ f4 mfma_tile(const AL &A, int mt, const h8 *b32, h4 b16)
{
    const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
    f4 acc;
    if (NC > 0)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(A.a32[mt][0], b32[0], zero, 0, 0, 0);
    else
        acc = __builtin_amdgcn_mfma_f32_16x16x16f16(A.a16[mt], b16, zero, 0, 0, 0);
#pragma unroll
    for (int ch = 1; ch < NC; ++ch)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(A.a32[mt][ch], b32[ch], acc, 0, 0, 0);
    if (NC > 0 && R16)
        acc += __builtin_amdgcn_mfma_f32_16x16x16f16(A.a16[mt], b16, zero, 0, 0, 0);
    return acc;
}

template <int KIN, int MOUT>
__device__ __forceinline__ void layer_from_regs(const LayerA<KIN, MOUT, true> &A,
                                                const Act<KIN> &in, Act<MOUT> &out)
{
    constexpr int NC = LayerA<KIN, MOUT, true>::NC, R16 = LayerA<KIN, MOUT, true>::R16;
    h8 b32[NC > 0 ? NC : 1];
    h4 b16 = {};
    // Each packed pair is one 32-bit register already in operand order, so
    // the operands are assembled whole (element-wise construction costs
    // shifts, ORs and permutes per half).
#pragma unroll
    for (int ch = 0; ch < NC; ++ch) {
        const f4 lo = in.acc[2 * ch], hi = in.acc[2 * ch + 1];
        const uint4 w = {h2_word(relu_pack(lo[0], lo[1])), h2_word(relu_pack(lo[2], lo[3])),
                         h2_word(relu_pack(hi[0], hi[1])), h2_word(relu_pack(hi[2], hi[3]))};
        b32[ch] = __builtin_bit_cast(h8, w);
    }
    if (R16) {
        const uint2 w = {h2_word(relu_pack(in.acc[0][0], in.acc[0][1])),
                         h2_word(relu_pack(in.acc[0][2], in.acc[0][3]))};
        b16 = __builtin_bit_cast(h4, w);
    }
#pragma unroll
    for (int mt = 0; mt < Act<MOUT>::MT; ++mt)
        out.acc[mt] = mfma_tile<NC, R16>(A, mt, b32, b16);
}

// First layer: B operand read from a [16][ld] fp16 tile (row = sample) in
// LDS or global memory.
template <int KIN, int MOUT>
__device__ __forceinline__ void layer_from_rows(const LayerA<KIN, MOUT, false> &A,
                                                const _Float16 *rows, int ld, int lane,
                                                Act<MOUT> &out)
{
    constexpr int NC = LayerA<KIN, MOUT, false>::NC, R16 = LayerA<KIN, MOUT, false>::R16;
    const int c = lane & 15, g = lane >> 4;
    const _Float16 *row = rows + c * ld;
    h8 b32[NC > 0 ? NC : 1];
    h4 b16 = {};
#pragma unroll
    for (int ch = 0; ch < NC; ++ch)
        b32[ch] = *(const h8 *)(row + ch * 32 + 8 * g);
    if (R16)
        b16 = *(const h4 *)(row + NC * 32 + 4 * g);
#pragma unroll
    for (int mt = 0; mt < Act<MOUT>::MT; ++mt)
        out.acc[mt] = mfma_tile<NC, R16>(A, mt, b32, b16);
}

// The whole MLP: IN -> HID (ReLU) -> [HID -> HID (ReLU)] x (NHID-1) -> 4.
template <int IN, int HID, int NHID>
struct MlpWeights {
    static_assert(NHID >= 1 && NHID <= 3, "1..3 hidden layers");
    LayerA<IN, HID, false> first;
    LayerA<HID, HID, true> mid[NHID > 1 ? NHID - 1 : 1];
    LayerA<HID, 4, true> head;

    // hl: the hidden width of the weights in W (at most HID; the layers are
    // [IN][hl], [hl][hl] x (NHID-1), [hl][4]).
    __device__ __forceinline__ void load(const _Float16 *W, int lane, int hl)
    {
        first.load(W, lane, IN, hl);
        const _Float16 *p = W + IN * hl;
#pragma unroll
        for (int m = 0; m < NHID - 1; ++m) {
            mid[m].load(p, lane, hl, hl);
            p += hl * hl;
        }
        head.load(p, lane, hl, 4);
    }
};

// Returns the raw head outputs: lanes 0..15 hold (sigma_raw, r, g, b) of
// sample column (lane & 15) in elements 0..3; other lanes hold padding.
template <int IN, int HID, int NHID>
__device__ __forceinline__ f4 mlp_tile(const MlpWeights<IN, HID, NHID> &Wt,
                                       const _Float16 *rows, int ld, int lane)
{
    Act<HID> a, b;
    layer_from_rows<IN, HID>(Wt.first, rows, ld, lane, a);
#pragma unroll
    for (int m = 0; m < NHID - 1; ++m) {
        layer_from_regs<HID, HID>(Wt.mid[m], a, b);
        a = b;
    }
    Act<4> o;
    layer_from_regs<HID, 4>(Wt.head, a, o);
    return o.acc[0];
}

// Output activations (Sec. 3.1): density exp(.), colour sigmoid(.), with the
// hardware exp2 and reciprocal (about 1 ulp).
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }
__device__ __forceinline__ float fast_sigmoid(float x)
{
    return __builtin_amdgcn_rcpf(1.0f + fast_exp(-x));
}

__device__ __forceinline__ float4 mlp_activate(f4 o)
{
    return make_float4(fast_exp(o[0]), fast_sigmoid(o[1]), fast_sigmoid(o[2]), fast_sigmoid(o[3]));
}

// --------------------------------------------------------------------------
// Eq. 1 front to back: alpha_k = 1 - exp(-sigma_k delta), the running
// transmittance excludes sample k, the remaining transmittance weights the
// background, and a ray stops once its transmittance is below t_term.
// A zero-length interval (delta = 0) has zero optical depth whatever sigma
// is: sigma delta is taken through max(., 0), which turns the inf * 0 of an
// overflowed density into 0 and leaves every other product unchanged
// (sigma = exp(.) >= 0).
// --------------------------------------------------------------------------
struct Composite {
    float r = 0.0f, g = 0.0f, b = 0.0f, T = 1.0f;

    __device__ __forceinline__ bool add(float4 s, float delta, float t_term)
    {
        const float alpha = 1.0f - fast_exp(-fmaxf(s.x * delta, 0.0f));
        const float w = T * alpha;
        r += w * s.y;
        g += w * s.z;
        b += w * s.w;
        T *= 1.0f - alpha;
        return T >= t_term;
    }

    __device__ __forceinline__ float4 finish(float bgr, float bgg, float bgb) const
    {
        return make_float4(r + T * bgr, g + T * bgg, b + T * bgb, 1.0f - T);
    }
};

}  // namespace mixrt
