/*
 * MixRT per-pixel rendering path -- plain CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no code, header, table or constant with the HIP
 * library: every step below is written out from its definition.
 *
 * Arithmetic is IEEE double, except the one place where a floating-point
 * value decides an integer: the grid cell of a hash-grid query is taken from
 * an fp32 product x*N_l, exactly as the GPU kernel takes it, so that voxel
 * corners and table indices can be compared bit for bit.
 *
 * Paper: "MixRT: Mixed Neural Representations For Real-Time NeRF Rendering"
 * (arXiv 2312.11841).  Steps of one pixel, in the paper's order:
 *   1. ray r = o + t d through the pixel                      (Sec. 3.1)
 *   2. ray-mesh hit p and texture coordinate p_t: read from a
 *      G-buffer, or found by testing the ray against every
 *      triangle of the mesh (the closest hit at t > 1e-4, equal
 *      t to the lower triangle index)                          (Fig. 2 step 1)
 *   3. calibrated point p_cali from the view-dependent
 *      displacement map                                        (Sec. 4.3.2, Eq. 2)
 *   4. K samples around p_cali, contracted into a ball of
 *      radius 2 (Mip-NeRF 360 contraction)                     (Sec. 2.1)
 *   5. multiresolution hash encoding: 8 grid vertices per
 *      level from a 1D hash table, trilinear interpolation,
 *      levels concatenated                                     (Sec. 3.1, 4.3.3, 5.1.2)
 *   6. small MLP -> density and colour                         (Sec. 3.1)
 *   7. volume rendering of the samples                         (Sec. 3.1, Eq. 1)
 *
 * Readings where the paper is silent or inconsistent:
 *   - Eq. 1 transmittance is exclusive of sample k; delta_k = delta for all k;
 *     the final transmittance blends a background colour.
 *   - Eq. 2, scalar form: the V channels are coefficients of the first V
 *     real spherical harmonics of d, their sum is a length along d (scale
 *     map 1).  Eq. 2 as printed (a 3-vector of SH sums times the scale map)
 *     and no displacement are the other two forms.
 *   - texels are addressed GL-style: centres at (i+0.5)/R, clamp to edge.
 *   - level resolutions N_l = floor(N_min b^l + 1e-6), b the geometric growth
 *     factor from N_min to N_max; dense indexing when (N_l+1)^3 <= T, else the
 *     XOR-of-primes spatial hash (1, 2654435761, 805459861) modulo T.
 *   - MLP without biases, ReLU hidden layers, outputs (sigma_raw, r, g, b),
 *     sigma = exp, rgb = sigmoid; with the MLP removed (Tab. 3), feature i
 *     is added to output i mod 4.
 *   - 8-bit maps stand for q_offset + q_scale * q.
 *   - the ray-mesh hit is sampled at the pixel centre, as rasterisation
 *     does; uv is the barycentric interpolation of the vertex uv.
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -fopenmp -shared -fPIC.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_PI 3.14159265358979323846

enum { ORC_F32 = 0, ORC_F16 = 1, ORC_U8 = 2 };

static int clampi(int v, int lo, int hi);

/* ------------------------------------------------------------------------ */
/* Stored values                                                              */
/* ------------------------------------------------------------------------ */

/* IEEE binary16 -> double, from the format's definition. */
double orc_half_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int expo = (h >> 10) & 31;
    int mant = h & 1023;
    double v;
    if (expo == 0)
        v = ldexp((double)mant, -24);                /* subnormal */
    else if (expo == 31)
        v = mant ? NAN : INFINITY;
    else
        v = ldexp((double)(mant + 1024), expo - 25); /* 1.m * 2^(e-15) */
    return sign ? -v : v;
}

static double load_value(const void *base, int dtype, int64_t i)
{
    switch (dtype) {
    case ORC_F32: return (double)((const float *)base)[i];
    case ORC_F16: return orc_half_to_double(((const uint16_t *)base)[i]);
    default: return NAN;
    }
}

/* ------------------------------------------------------------------------ */
/* Multiresolution grid: level resolutions                                    */
/* ------------------------------------------------------------------------ */

/* Geometric progression from N_min to N_max over L levels (Instant-NGP's
 * schedule, which the paper follows); the 1e-6 guard keeps N_0 = N_min and
 * N_{L-1} = N_max exact despite rounding in b^l. */
int orc_level_resolutions(int L, int n_min, int n_max, int32_t *out)
{
    if (L < 1 || n_min < 1 || n_max < n_min)
        return -1;
    if (L == 1) {
        out[0] = n_min;
        return 0;
    }
    double b = exp((log((double)n_max) - log((double)n_min)) / (double)(L - 1));
    for (int l = 0; l < L; ++l)
        out[l] = (int32_t)floor((double)n_min * pow(b, (double)l) + 1e-6);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Real spherical harmonics (orthonormal, no Condon-Shortley phase)           */
/* ------------------------------------------------------------------------ */

static double factorial(int n)
{
    double r = 1.0;
    for (int i = 2; i <= n; ++i)
        r *= (double)i;
    return r;
}

/* Associated Legendre function P_l^m(x), m >= 0, without the (-1)^m phase:
 * P_m^m = (2m-1)!! (1-x^2)^{m/2}, P_{m+1}^m = x (2m+1) P_m^m,
 * (l-m) P_l^m = (2l-1) x P_{l-1}^m - (l+m-1) P_{l-2}^m. */
static double assoc_legendre(int l, int m, double x)
{
    double pmm = 1.0;
    double s = sqrt(fmax(0.0, 1.0 - x * x));
    for (int i = 1; i <= m; ++i)
        pmm *= (double)(2 * i - 1) * s;
    if (l == m)
        return pmm;
    double pm1 = x * (double)(2 * m + 1) * pmm;
    if (l == m + 1)
        return pm1;
    double pl = 0.0;
    for (int ll = m + 2; ll <= l; ++ll) {
        pl = ((double)(2 * ll - 1) * x * pm1 - (double)(ll + m - 1) * pmm) / (double)(ll - m);
        pmm = pm1;
        pm1 = pl;
    }
    return pl;
}

/* Y_l^m(d) for a unit vector d = (x, y, z): polar angle from +z, azimuth
 * atan2(y, x); m > 0 takes cos(m phi), m < 0 takes sin(|m| phi). */
double orc_sh_real(int l, int m, double x, double y, double z)
{
    int am = m < 0 ? -m : m;
    double k = sqrt((2.0 * l + 1.0) / (4.0 * ORC_PI) * factorial(l - am) / factorial(l + am));
    double ct = z > 1.0 ? 1.0 : (z < -1.0 ? -1.0 : z);
    double p = assoc_legendre(l, am, ct);
    if (m == 0)
        return k * p;
    double phi = atan2(y, x);
    if (m > 0)
        return sqrt(2.0) * k * p * cos((double)am * phi);
    return sqrt(2.0) * k * p * sin((double)am * phi);
}

/* First n functions in the order (l, m = -l..l), l = 0, 1, 2, ... */
void orc_sh_basis(int n, const double *d, double *out)
{
    int v = 0;
    for (int l = 0; v < n; ++l)
        for (int m = -l; m <= l && v < n; ++m)
            out[v++] = orc_sh_real(l, m, d[0], d[1], d[2]);
}

/* ------------------------------------------------------------------------ */
/* Step 1: camera ray (Sec. 3.1)                                              */
/* ------------------------------------------------------------------------ */

/* cam: c2w row-major 3x4 (12), vertical fov in degrees, background rgb.
 * Pinhole with OpenGL axes: looks down -z, +y up, pixel (i, j) with row 0 at
 * the top, sampled through its centre. */
void orc_camera_ray(const float *cam, int W, int H, int i, int j, double *o, double *d)
{
    double f = 0.5 * (double)H / tan(0.5 * (double)cam[12] * ORC_PI / 180.0);
    double dc[3] = {((double)i + 0.5 - 0.5 * W) / f, -((double)j + 0.5 - 0.5 * H) / f, -1.0};
    double n2 = 0.0;
    for (int r = 0; r < 3; ++r) {
        d[r] = (double)cam[4 * r + 0] * dc[0] + (double)cam[4 * r + 1] * dc[1] +
               (double)cam[4 * r + 2] * dc[2];
        o[r] = (double)cam[4 * r + 3];
        n2 += d[r] * d[r];
    }
    double inv = 1.0 / sqrt(n2);
    for (int r = 0; r < 3; ++r)
        d[r] *= inv;
}

/* ------------------------------------------------------------------------ */
/* Step 3: displacement texture fetch and calibration (Eq. 2)                 */
/* ------------------------------------------------------------------------ */

static int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

/* A displacement-map texture: [R][R][C] values of one dtype; 8-bit values
 * stand for q_offset + q_scale * q (the maps are quantised to 8 bits after
 * training, Sec. 4.3.2). */
typedef struct {
    int R, C, dtype;
    const void *data;
    double q_scale, q_offset;
} orc_map;

static double map_value(const orc_map *m, int64_t i)
{
    if (m->dtype == ORC_U8)
        return m->q_offset + m->q_scale * (double)((const uint8_t *)m->data)[i];
    return load_value(m->data, m->dtype, i);
}

/* Bilinear fetch of the first nch channels of a map at (u, v). */
static void map_bilinear(const orc_map *m, int nch, double u, double v, double *out)
{
    const int R = m->R;
    double a = u * R - 0.5, b = v * R - 0.5;
    double fa = floor(a), fb = floor(b);
    double wa = a - fa, wb = b - fb;
    int i0 = (int)fa, j0 = (int)fb;
    int ia[2] = {clampi(i0, 0, R - 1), clampi(i0 + 1, 0, R - 1)};
    int jb[2] = {clampi(j0, 0, R - 1), clampi(j0 + 1, 0, R - 1)};
    double w[2][2] = {{(1 - wa) * (1 - wb), wa * (1 - wb)}, {(1 - wa) * wb, wa * wb}};
    for (int c = 0; c < nch; ++c) {
        double s = 0.0;
        for (int y = 0; y < 2; ++y)
            for (int x = 0; x < 2; ++x)
                s += w[y][x] * map_value(m, ((int64_t)jb[y] * R + ia[x]) * m->C + c);
        out[c] = s;
    }
}

/* Bilinear fetch of the V channels of an [R][R][V] texture at (u, v). */
void orc_tex_bilinear(const void *tex, int dtype, int R, int V, double u, double v, double *out)
{
    orc_map m = {R, V, dtype, tex, 0.0, 0.0};
    map_bilinear(&m, V, u, v, out);
}

/* The same for a map with C stored channels and 8-bit dequantisation. */
void orc_map_bilinear(const void *data, int dtype, int R, int C, int nch, double q_scale,
                      double q_offset, double u, double v, double *out)
{
    orc_map m = {R, C, dtype, data, q_scale, q_offset};
    map_bilinear(&m, nch, u, v, out);
}

/* p_cali = p + S(m(p_t), d) d : the SH-weighted sum of the texture channels
 * is a signed length along the view direction. */
void orc_calibrate(const double *p, const double *d, const double *m, int V, double *p_cali)
{
    double y[64];
    orc_sh_basis(V, d, y);
    double s = 0.0;
    for (int c = 0; c < V; ++c)
        s += y[c] * m[c];
    for (int r = 0; r < 3; ++r)
        p_cali[r] = p[r] + s * d[r];
}

/* Eq. 2 as printed: p_cali = p + S(m_SH(p_t), d) * m_s(p_t), where the SH map
 * holds, for each of the 3 axes, the coefficients of the first nb real
 * harmonics of d (channel a*nb + v), and m_s is the scalar scale map. */
void orc_calibrate_vec3(const double *p, const double *d, const double *m, int nb, double ms,
                        double *p_cali)
{
    double y[64];
    orc_sh_basis(nb, d, y);
    for (int a = 0; a < 3; ++a) {
        double s = 0.0;
        for (int v = 0; v < nb; ++v)
            s += y[v] * m[a * nb + v];
        p_cali[a] = p[a] + s * ms;
    }
}

/* ------------------------------------------------------------------------ */
/* Step 4: scene contraction and normalisation to the unit cube (Sec. 2.1)    */
/* ------------------------------------------------------------------------ */

void orc_contract(const double *q, double *x)
{
    double r = sqrt(q[0] * q[0] + q[1] * q[1] + q[2] * q[2]);
    for (int a = 0; a < 3; ++a) {
        double c = r <= 1.0 ? q[a] : (2.0 - 1.0 / r) * (q[a] / r);
        double u = (c + 2.0) / 4.0;
        x[a] = u < 0.0 ? 0.0 : (u > 1.0 ? 1.0 : u);
    }
}

/* ------------------------------------------------------------------------ */
/* Step 5: multiresolution hash encoding (Sec. 3.1, 4.3.3)                    */
/* ------------------------------------------------------------------------ */

static uint32_t grid_index(const int32_t v[3], int32_t N, uint64_t T)
{
    uint64_t side = (uint64_t)N + 1;
    if (side * side * side <= T)  /* the level fits: one entry per vertex */
        return (uint32_t)((uint64_t)v[0] + side * (uint64_t)v[1] + side * side * (uint64_t)v[2]);
    uint32_t h = ((uint32_t)v[0] * 1u) ^ ((uint32_t)v[1] * 2654435761u) ^ ((uint32_t)v[2] * 805459861u);
    return h & (uint32_t)(T - 1);
}

/* One level of one query.  x: fp32 position in [0,1]^3.  Writes the lower
 * voxel corner, the 8 table indices and trilinear weights (corner beta has
 * offset (beta&1, beta>>1&1, beta>>2&1)) and the F interpolated features. */
void orc_hash_level(const float *x, int32_t N, int log2T, int F, int tdtype,
                    const void *table_level, int32_t *corner, uint32_t *idx,
                    double *w, double *feat)
{
    uint64_t T = (uint64_t)1 << log2T;
    float pos[3];
    int32_t c0[3];
    double fr[3];
    for (int a = 0; a < 3; ++a) {
        pos[a] = x[a] * (float)N;                /* one fp32 rounding */
        int32_t c = (int32_t)floorf(pos[a]);
        c0[a] = c < 0 ? 0 : (c > N - 1 ? N - 1 : c);
        fr[a] = (double)pos[a] - (double)c0[a];
        corner[a] = c0[a];
    }
    for (int f = 0; f < F; ++f)
        feat[f] = 0.0;
    for (int beta = 0; beta < 8; ++beta) {
        int32_t v[3];
        double wt = 1.0;
        for (int a = 0; a < 3; ++a) {
            int bit = (beta >> a) & 1;
            v[a] = c0[a] + bit;
            wt *= bit ? fr[a] : 1.0 - fr[a];
        }
        uint32_t id = grid_index(v, N, T);
        idx[beta] = id;
        w[beta] = wt;
        for (int f = 0; f < F; ++f)
            feat[f] += wt * load_value(table_level, tdtype, (int64_t)id * F + f);
    }
}

/* n queries x[n][3] (fp32) through all L levels of table [L][T][F].
 * Outputs (any may be NULL): corner [n][L][3], idx [n][L][8], w [n][L][8],
 * feat [n][L*F] (level-major). */
int orc_hash_encode(int64_t n, const float *x, int L, int n_min, int n_max, int log2T,
                    int F, int tdtype, const void *table, int32_t *corner, uint32_t *idx,
                    double *w, double *feat)
{
    int32_t Nl[64];
    if (L > 64 || orc_level_resolutions(L, n_min, n_max, Nl))
        return -1;
    int64_t T = (int64_t)1 << log2T;
    size_t esz = tdtype == ORC_F32 ? 4 : 2;
    for (int64_t s = 0; s < n; ++s) {
        for (int l = 0; l < L; ++l) {
            int32_t c[3];
            uint32_t id[8];
            double wt[8], ft[16];
            const char *lev = (const char *)table + (size_t)l * (size_t)T * (size_t)F * esz;
            orc_hash_level(x + 3 * s, Nl[l], log2T, F, tdtype, lev, c, id, wt, ft);
            if (corner)
                memcpy(corner + (s * L + l) * 3, c, sizeof c);
            if (idx)
                memcpy(idx + (s * L + l) * 8, id, sizeof id);
            if (w)
                memcpy(w + (s * L + l) * 8, wt, sizeof wt);
            if (feat)
                for (int f = 0; f < F; ++f)
                    feat[s * L * F + l * F + f] = ft[f];
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Step 6: the small MLP (Sec. 3.1)                                           */
/* ------------------------------------------------------------------------ */

/* widths[0..n_layers]: layer m maps widths[m] -> widths[m+1] with fp16
 * weights stored row-major [in][out], layers concatenated.  Hidden layers use
 * ReLU; the 4 outputs become sigma = exp(o0), rgb = 1/(1+exp(-o1..3)). */
int orc_mlp(int64_t n, const double *in, int n_layers, const int32_t *widths,
            const uint16_t *weights, double *out4)
{
    if (n_layers == 0) {
        /* The MLP removed (the ablation of Tab. 3): the inputs are summed per
         * component, input i feeding output i mod 4 = (sigma_raw, r, g, b). */
        if (widths[0] < 4 || widths[0] % 4)
            return -1;
        for (int64_t s = 0; s < n; ++s) {
            double o[4] = {0.0, 0.0, 0.0, 0.0};
            for (int i = 0; i < widths[0]; ++i)
                o[i % 4] += in[s * widths[0] + i];
            out4[4 * s + 0] = exp(o[0]);
            for (int c = 1; c < 4; ++c)
                out4[4 * s + c] = 1.0 / (1.0 + exp(-o[c]));
        }
        return 0;
    }
    if (n_layers < 1 || widths[n_layers] != 4)
        return -1;
    int maxw = 0;
    for (int m = 0; m <= n_layers; ++m)
        if (widths[m] > maxw)
            maxw = widths[m];
    double *a = (double *)malloc(sizeof(double) * maxw);
    double *b = (double *)malloc(sizeof(double) * maxw);
    for (int64_t s = 0; s < n; ++s) {
        memcpy(a, in + s * widths[0], sizeof(double) * widths[0]);
        const uint16_t *wm = weights;
        for (int m = 0; m < n_layers; ++m) {
            int ni = widths[m], no = widths[m + 1];
            for (int o = 0; o < no; ++o) {
                double acc = 0.0;
                for (int k = 0; k < ni; ++k)
                    acc += orc_half_to_double(wm[(int64_t)k * no + o]) * a[k];
                b[o] = (m < n_layers - 1 && acc < 0.0) ? 0.0 : acc;
            }
            wm += (int64_t)ni * no;
            memcpy(a, b, sizeof(double) * no);
        }
        out4[4 * s + 0] = exp(a[0]);
        for (int c = 1; c < 4; ++c)
            out4[4 * s + c] = 1.0 / (1.0 + exp(-a[c]));
    }
    free(a);
    free(b);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Step 7: volume rendering (Eq. 1)                                           */
/* ------------------------------------------------------------------------ */

/* srgb [rays][K][4] = (sigma, r, g, b); bg [rays][3].  The transmittance of
 * sample k is exp(-sum_{j<k} sigma_j delta); the transmittance left after the
 * last sample weights the background.  out [rays][4] = (rgb, alpha).
 * A sample's optical depth sigma_k delta is 0 when delta = 0: an interval of
 * zero length absorbs nothing, whatever the density (this also defines the
 * product for a density that overflowed to infinity). */
void orc_composite(int64_t rays, int K, const double *srgb, double delta, const double *bg,
                   double *out)
{
    for (int64_t r = 0; r < rays; ++r) {
        const double *s = srgb + r * K * 4;
        double c[3] = {0.0, 0.0, 0.0};
        double optical = 0.0;  /* sum_{j<k} sigma_j delta */
        for (int k = 0; k < K; ++k) {
            double T = exp(-optical);
            double tau = delta > 0.0 ? s[4 * k] * delta : 0.0;
            double alpha = 1.0 - exp(-tau);
            for (int ch = 0; ch < 3; ++ch)
                c[ch] += T * alpha * s[4 * k + 1 + ch];
            optical += tau;
        }
        double Tend = exp(-optical);
        for (int ch = 0; ch < 3; ++ch)
            out[4 * r + ch] = c[ch] + Tend * bg[3 * r + ch];
        out[4 * r + 3] = 1.0 - Tend;
    }
}

/* ------------------------------------------------------------------------ */
/* The whole path for a list of pixels                                        */
/* ------------------------------------------------------------------------ */

typedef struct {
    int views, H, W;
    const float *g0;         /* [views][H][W][4]: t, u, v, - */
    const float *cams;       /* [views][16]: c2w 3x4, fov_y_deg, bg rgb */
    int tex_R, tex_V, tex_dtype;
    const void *tex;         /* [R][R][V] */
    int L, log2T, F, n_min, n_max, table_dtype;
    const void *table;       /* [L][T][F] */
    int n_layers;
    const int32_t *widths;   /* n_layers + 1 */
    int view_sh_dim;         /* 0 or 16 */
    const uint16_t *weights; /* concatenated [in][out] fp16 */
    int K;
    double delta;
    /* displacement form: 0 scalar along the ray (tex_V channels), 1 Eq. 2's
     * vector times scale (3 (sh_degree+1)^2 channels + the scale map), 2 none */
    int disp_mode;
    int tex_C;               /* stored channels per texel (>= used) */
    int sh_degree;
    const void *scale;       /* [R][R] scale map (mode 1) */
    double q_scale[2], q_offset[2]; /* 8-bit maps: [0] coefficients, [1] scale */
} orc_scene;

/* Steps 1-4 for one pixel.  Returns 0 for a miss (no samples).  x receives K
 * fp32-rounded cube positions (the hash grid's input), d the unit ray
 * direction, bg the camera's background. */
static int pixel_samples(const orc_scene *sc, int64_t pix, float *x, double *xd, double *d,
                         double *bg)
{
    int64_t hw = (int64_t)sc->H * sc->W;
    int view = (int)(pix / hw);
    int64_t rem = pix % hw;
    int j = (int)(rem / sc->W), i = (int)(rem % sc->W);
    const float *cam = sc->cams + 16 * view;
    for (int c = 0; c < 3; ++c)
        bg[c] = cam[13 + c];
    double o[3];
    orc_camera_ray(cam, sc->W, sc->H, i, j, o, d);
    const float *g = sc->g0 + 4 * pix;
    double t = g[0];
    if (!(t > 0.0 && isfinite(t)))
        return 0;
    double p[3], m[64], pc[3];
    for (int r = 0; r < 3; ++r)
        p[r] = o[r] + t * d[r];
    orc_map coef = {sc->tex_R, sc->tex_C, sc->tex_dtype, sc->tex, sc->q_scale[0], sc->q_offset[0]};
    if (sc->disp_mode == 0) {
        map_bilinear(&coef, sc->tex_V, g[1], g[2], m);
        orc_calibrate(p, d, m, sc->tex_V, pc);
    } else if (sc->disp_mode == 1) {
        int nb = (sc->sh_degree + 1) * (sc->sh_degree + 1);
        orc_map sm = {sc->tex_R, 1, sc->tex_dtype, sc->scale, sc->q_scale[1], sc->q_offset[1]};
        double ms;
        map_bilinear(&coef, 3 * nb, g[1], g[2], m);
        map_bilinear(&sm, 1, g[1], g[2], &ms);
        orc_calibrate_vec3(p, d, m, nb, ms, pc);
    } else {
        for (int r = 0; r < 3; ++r)
            pc[r] = p[r];
    }
    for (int k = 0; k < sc->K; ++k) {
        double off = ((double)k - 0.5 * (double)(sc->K - 1)) * sc->delta;
        double q[3], xc[3];
        for (int r = 0; r < 3; ++r)
            q[r] = pc[r] + off * d[r];
        orc_contract(q, xc);
        for (int r = 0; r < 3; ++r) {
            if (xd)
                xd[3 * k + r] = xc[r];
            x[3 * k + r] = (float)xc[r];
        }
    }
    return 1;
}

static void render_one(const orc_scene *sc, int64_t pix, double *out)
{
    int K = sc->K, L = sc->L, F = sc->F;
    int in_w = sc->widths[0];
    float *x = (float *)malloc(sizeof(float) * 3 * K);
    double *h = (double *)malloc(sizeof(double) * in_w * K);
    double *srgb = (double *)malloc(sizeof(double) * 4 * K);
    double d[3], bg[3];
    if (!pixel_samples(sc, pix, x, NULL, d, bg)) {
        for (int c = 0; c < 3; ++c)
            out[c] = bg[c];
        out[3] = 0.0;
    } else {
        double sh[16];
        if (sc->view_sh_dim)
            orc_sh_basis(sc->view_sh_dim, d, sh);
        for (int k = 0; k < K; ++k) {
            double *hk = h + (int64_t)k * in_w;
            orc_hash_encode(1, x + 3 * k, L, sc->n_min, sc->n_max, sc->log2T, F,
                            sc->table_dtype, sc->table, NULL, NULL, NULL, hk);
            for (int e = 0; e < sc->view_sh_dim; ++e)
                hk[L * F + e] = sh[e];
        }
        orc_mlp(K, h, sc->n_layers, sc->widths, sc->weights, srgb);
        orc_composite(1, K, srgb, sc->delta, bg, out);
    }
    free(x);
    free(h);
    free(srgb);
}

int orc_render_pixels(const orc_scene *sc, int64_t n_pix, const int64_t *pix, double *out,
                      int n_threads)
{
    if (sc->widths[0] != sc->L * sc->F + sc->view_sh_dim || sc->tex_V > 64 ||
        sc->view_sh_dim > 16 || sc->F > 16 || sc->sh_degree > 3 ||
        (sc->disp_mode == 0 && sc->tex_C < sc->tex_V) ||
        (sc->disp_mode == 1 && sc->tex_C < 3 * (sc->sh_degree + 1) * (sc->sh_degree + 1)))
        return -1;
#ifdef _OPENMP
    if (n_threads < 1)
        n_threads = 1;
#pragma omp parallel for schedule(dynamic, 64) num_threads(n_threads)
#endif
    for (int64_t q = 0; q < n_pix; ++q)
        render_one(sc, pix[q], out + 4 * q);
    return 0;
}

/* Steps 1-4 only: per pixel, K fp32 cube positions [n_pix][K][3] (the value
 * fed to the grid), their double values, and a hit flag. */
int orc_pixel_samples(const orc_scene *sc, int64_t n_pix, const int64_t *pix, float *x,
                      double *xd, int32_t *hit)
{
    for (int64_t q = 0; q < n_pix; ++q) {
        double d[3], bg[3];
        int ok = pixel_samples(sc, pix[q], x + 3 * sc->K * q, xd ? xd + 3 * sc->K * q : NULL, d,
                               bg);
        hit[q] = ok;
        if (!ok)
            for (int k = 0; k < 3 * sc->K; ++k) {
                x[3 * sc->K * q + k] = 0.0f;
                if (xd)
                    xd[3 * sc->K * q + k] = 0.0;
            }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Step 2's input: the coarse-mesh hit per pixel (Fig. 2 step 1)              */
/* ------------------------------------------------------------------------ */

/* Moller-Trumbore in double for triangle f: writes t, the barycentrics
 * (b1, b2) of corners 1 and 2 and the cosine between d and the face normal;
 * returns 0 when the ray is parallel to it. */
int orc_ray_triangle(const double *o, const double *d, const float *pos, const int32_t *faces,
                     int64_t f, double *t, double *b1, double *b2, double *cosine)
{
    const float *a = pos + 3 * (int64_t)faces[3 * f];
    const float *b = pos + 3 * (int64_t)faces[3 * f + 1];
    const float *c = pos + 3 * (int64_t)faces[3 * f + 2];
    double e1[3], e2[3], s[3], p[3], q[3];
    for (int k = 0; k < 3; ++k) {
        e1[k] = (double)b[k] - (double)a[k];
        e2[k] = (double)c[k] - (double)a[k];
        s[k] = o[k] - (double)a[k];
    }
    p[0] = d[1] * e2[2] - d[2] * e2[1];
    p[1] = d[2] * e2[0] - d[0] * e2[2];
    p[2] = d[0] * e2[1] - d[1] * e2[0];
    double det = e1[0] * p[0] + e1[1] * p[1] + e1[2] * p[2];
    if (fabs(det) < 1e-300)
        return 0;
    double n[3] = {e1[1] * e2[2] - e1[2] * e2[1], e1[2] * e2[0] - e1[0] * e2[2],
                   e1[0] * e2[1] - e1[1] * e2[0]};
    *cosine = -det / sqrt(n[0] * n[0] + n[1] * n[1] + n[2] * n[2]);  /* det = -d.n */
    double inv = 1.0 / det;
    q[0] = s[1] * e1[2] - s[2] * e1[1];
    q[1] = s[2] * e1[0] - s[0] * e1[2];
    q[2] = s[0] * e1[1] - s[1] * e1[0];
    *b1 = (s[0] * p[0] + s[1] * p[1] + s[2] * p[2]) * inv;
    *b2 = (d[0] * q[0] + d[1] * q[1] + d[2] * q[2]) * inv;
    *t = (e2[0] * q[0] + e2[1] * q[1] + e2[2] * q[2]) * inv;
    return 1;
}

/* Closest intersection of the ray o + t d (t > t_min) with every triangle of
 * a mesh (brute force); equal t goes to the lower triangle index.  Returns the
 * triangle (-1 for a miss) and writes t, the barycentrics (b1, b2) of corners
 * 1 and 2, the interpolated vertex uv, the unit face normal e1 x e2, and
 * *ambiguous = 1 when a fp32 solver may legitimately answer otherwise: the
 * hit lies within eps_b of an edge (barycentric margin), or another triangle
 * that is hit or nearly hit (margin > -eps_b) lies no farther than
 * t (1 + eps_t); for a miss, when any triangle in front is nearly hit.  Both
 * slacks widen as 0.1 / |cos| below a cosine of 0.1, since a grazing ray's
 * rounding error grows like the inverse cosine. */
static double graze(double cosine)
{
    return fmax(1.0, 0.1 / fmax(fabs(cosine), 1e-12));
}

int64_t orc_ray_mesh(const double *o, const double *d, const float *pos, const int32_t *faces,
                     int64_t nf, const float *uv, double t_min, double *t_out, double *bary,
                     double *uv_out, double *normal, int *ambiguous)
{
    const double eps_b = 2e-4, eps_t = 1e-4;
    double best = INFINITY, bb1 = 0.0, bb2 = 0.0, bcos = 1.0, t, b1, b2, cs;
    int64_t best_i = -1;
    for (int64_t f = 0; f < nf; ++f) {
        if (!orc_ray_triangle(o, d, pos, faces, f, &t, &b1, &b2, &cs))
            continue;
        if (t > t_min && b1 >= 0.0 && b2 >= 0.0 && b1 + b2 <= 1.0 && t < best) {
            best = t;              /* strict: an equal t keeps the lower index */
            best_i = f;
            bb1 = b1;
            bb2 = b2;
            bcos = cs;
        }
    }
    *ambiguous = best_i >= 0 && fmin(fmin(bb1, bb2), 1.0 - bb1 - bb2) < eps_b * graze(bcos);
    for (int64_t f = 0; f < nf && !*ambiguous; ++f) {
        if (f == best_i || !orc_ray_triangle(o, d, pos, faces, f, &t, &b1, &b2, &cs))
            continue;
        double g = graze(cs) * (best_i >= 0 ? graze(bcos) : 1.0);
        double reach = best_i >= 0 ? best * (1.0 + eps_t * g) : INFINITY;
        if (t > t_min && t <= reach && fmin(fmin(b1, b2), 1.0 - b1 - b2) > -eps_b * g)
            *ambiguous = 1;
    }
    if (best_i < 0)
        return -1;
    const int32_t *fc = faces + 3 * best_i;
    double b0 = 1.0 - bb1 - bb2, e1[3], e2[3];
    for (int k = 0; k < 3; ++k) {
        e1[k] = (double)pos[3 * fc[1] + k] - (double)pos[3 * fc[0] + k];
        e2[k] = (double)pos[3 * fc[2] + k] - (double)pos[3 * fc[0] + k];
    }
    double n[3] = {e1[1] * e2[2] - e1[2] * e2[1], e1[2] * e2[0] - e1[0] * e2[2],
                   e1[0] * e2[1] - e1[1] * e2[0]};
    double nn = sqrt(n[0] * n[0] + n[1] * n[1] + n[2] * n[2]);
    for (int k = 0; k < 3; ++k)
        normal[k] = nn > 0.0 ? n[k] / nn : 0.0;
    for (int k = 0; k < 2; ++k)
        uv_out[k] = uv ? b0 * uv[2 * fc[0] + k] + bb1 * uv[2 * fc[1] + k] + bb2 * uv[2 * fc[2] + k]
                       : 0.0;
    *t_out = best;
    bary[0] = bb1;
    bary[1] = bb2;
    return best_i;
}

/* The G-buffer of a list of pixels of views x H x W cameras (cams [views][16]):
 * per pixel g0 = (t, u, v, 0) (t = -1 for a miss), normal [3], triangle id
 * (-1 miss) and the ambiguity flag. */
int orc_raycast_pixels(int views, int H, int W, const float *cams, const float *pos,
                       const int32_t *faces, int64_t nf, const float *uv, int64_t n_pix,
                       const int64_t *pix, double *g0, double *normal, int64_t *tri, int32_t *amb,
                       int n_threads)
{
    (void)views;
#ifdef _OPENMP
    if (n_threads < 1)
        n_threads = 1;
#pragma omp parallel for schedule(dynamic, 4) num_threads(n_threads)
#endif
    for (int64_t q = 0; q < n_pix; ++q) {
        int64_t hw = (int64_t)H * W;
        int view = (int)(pix[q] / hw);
        int64_t rem = pix[q] % hw;
        int j = (int)(rem / W), i = (int)(rem % W);
        double o[3], d[3], t, bary[2], uvo[2], n[3];
        int ambiguous = 0;
        orc_camera_ray(cams + 16 * view, W, H, i, j, o, d);
        int64_t f = orc_ray_mesh(o, d, pos, faces, nf, uv, 1e-4, &t, bary, uvo, n, &ambiguous);
        tri[q] = f;
        amb[q] = ambiguous;
        g0[4 * q + 0] = f < 0 ? -1.0 : t;
        g0[4 * q + 1] = f < 0 ? 0.0 : uvo[0];
        g0[4 * q + 2] = f < 0 ? 0.0 : uvo[1];
        g0[4 * q + 3] = 0.0;
        for (int k = 0; k < 3; ++k)
            normal[3 * q + k] = f < 0 ? 0.0 : n[k];
    }
    return 0;
}

int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
