// C ABI of the MixRT per-pixel rendering library (declared in include/mixrt.h).
//
// Host side: descriptor validation (pure host code, no HIP call), the level
// resolution table, camera constants, and the launches of the kernels in
// mixrt_render.hip and mixrt_stages.hip on the context's stream; the mesh
// objects of the geometry stage (arrays built in mixrt_mesh.cpp, kernels in
// mixrt_raster.hip and mixrt_raycast.hip).
#include "mixrt.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <atomic>
#include <mutex>
#include <new>
#include <string>

#include "mixrt_common.hpp"
#include "mixrt_launch.hpp"
#include "mixrt_mesh.hpp"

struct mixrt_ctx {
    int device = 0;
    hipStream_t stream = nullptr;
    uint32_t flags = 0;
    int32_t tile_stripe = 0;
    int32_t early_stop_chunk = 0;
    int32_t block_levels = 0;
    unsigned int *work = nullptr;   // device: the render kernels' work counters
    int cus = 0;
    int64_t l2_bytes = 0;
    std::string err;
};

// The work counters of mixrt_render_noalloc: one array per device (each
// device holds its own copy), found with hipGetSymbolAddress at set-up.
static __device__ __align__(256) unsigned int scratch[mixrt::kWorkWords];
static_assert(sizeof(scratch) == MIXRT_NOALLOC_SCRATCH_BYTES, "scratch size");

struct mixrt_mesh {
    int device = 0;
    void *mem = nullptr;           // one device allocation holding every array
    mixrt::MeshGridK k{};
    mixrt_mesh_info info{};
};

namespace {

thread_local std::string t_err;

// Device address of `scratch` on each device that a context was created on
// (null: not set up).  In host code the array's name stands for a host-side
// handle, never a device address: kernels get these pointers.
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
std::atomic<unsigned int *> g_scratch[kMaxScratchDevices];

// Once per device, with that device current: look up the array's address
// and zero it.  Returns a HIP error; the device keeps no address on failure.
hipError_t scratch_setup(int device)
{
    if (device < 0 || device >= kMaxScratchDevices) return hipSuccess;  // no no-alloc path
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch[device].load()) return hipSuccess;
    unsigned int *ptr = nullptr;
    hipError_t e = hipGetSymbolAddress((void **)&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    e = hipMemset(ptr, 0, sizeof(scratch));
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return e;
    g_scratch[device].store(ptr);
    return hipSuccess;
}

int fail(mixrt_ctx *ctx, int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_err = buf;
    if (ctx) ctx->err = buf;
    return code;
}

void clear_err(mixrt_ctx *ctx)
{
    t_err.clear();
    if (ctx) ctx->err.clear();
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// Level resolutions: geometric progression from N_min to N_max, floor with a
// 1e-6 guard so that the end points are exact.
void level_table(int L, int n_min, int n_max, int32_t *out)
{
    if (L == 1) {
        out[0] = n_min;
        return;
    }
    const double growth = std::exp((std::log((double)n_max) - std::log((double)n_min)) / (L - 1));
    for (int l = 0; l < L; ++l)
        out[l] = (int32_t)std::floor((double)n_min * std::pow(growth, (double)l) + 1e-6);
}

struct Msg {
    char *buf;
    size_t cap;
};

int vfail(Msg m, int code, const char *fmt, ...)
{
    char tmp[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(tmp, sizeof tmp, fmt, ap);
    va_end(ap);
    if (m.buf && m.cap) {
        strncpy(m.buf, tmp, m.cap - 1);
        m.buf[m.cap - 1] = 0;
    }
    return code;
}

int check_cams(const mixrt_camera *cams, int views, Msg m)
{
    if (!cams) return vfail(m, MIXRT_EINVAL, "cams is NULL");
    for (int v = 0; v < views; ++v) {
        const mixrt_camera &c = cams[v];
        if (!(c.fov_y_deg > 0.0f && c.fov_y_deg < 180.0f))
            return vfail(m, MIXRT_EINVAL, "cams[%d].fov_y_deg=%g outside (0,180)", v, c.fov_y_deg);
        for (int i = 0; i < 12; ++i)
            if (!std::isfinite(c.c2w[i]))
                return vfail(m, MIXRT_EINVAL, "cams[%d].c2w has a non-finite entry", v);
    }
    return MIXRT_OK;
}

int check_gbuf(const mixrt_gbuffer *g, const mixrt_camera *cams, Msg m)
{
    if (!g) return vfail(m, MIXRT_EINVAL, "gbuf is NULL");
    if (g->views < 1 || g->views > MIXRT_MAX_VIEWS)
        return vfail(m, MIXRT_EINVAL, "gbuf.views=%d outside 1..%d", g->views, MIXRT_MAX_VIEWS);
    if (g->W < 1 || g->H < 1) return vfail(m, MIXRT_EINVAL, "gbuf W=%d H=%d", g->W, g->H);
    if ((int64_t)g->views * g->H * g->W >= ((int64_t)1 << 31))
        return vfail(m, MIXRT_EUNSUPPORTED, "more than 2^31-1 pixels per call");
    if (!g->g0) return vfail(m, MIXRT_EINVAL, "gbuf.g0 is NULL");
    if (!aligned16(g->g0)) return vfail(m, MIXRT_EINVAL, "gbuf.g0 not 16-byte aligned");
    return check_cams(cams, g->views, m);
}

int disp_channels(const mixrt_disp_tex *d)
{
    if (d->mode == MIXRT_DISP_ALONG_RAY) return d->V;
    if (d->mode == MIXRT_DISP_SH_VEC3) return 3 * (d->sh_degree + 1) * (d->sh_degree + 1);
    return 0;
}

int stored_channels(const mixrt_disp_tex *d) { return d->C > 0 ? d->C : disp_channels(d); }

int check_disp(const mixrt_disp_tex *d, Msg m)
{
    if (!d) return vfail(m, MIXRT_EINVAL, "disp is NULL");
    if (d->mode != MIXRT_DISP_ALONG_RAY && d->mode != MIXRT_DISP_SH_VEC3 &&
        d->mode != MIXRT_DISP_NONE)
        return vfail(m, MIXRT_EUNSUPPORTED, "disp.mode=%d", d->mode);
    if (d->mode == MIXRT_DISP_NONE) return MIXRT_OK;
    if (d->R < 1 || d->R > (1 << 15)) return vfail(m, MIXRT_EINVAL, "disp.R=%d", d->R);
    if (d->mode == MIXRT_DISP_ALONG_RAY && (d->V < 1 || d->V > MIXRT_MAX_TEX_CHANNELS))
        return vfail(m, MIXRT_EUNSUPPORTED, "disp.V=%d outside 1..%d", d->V, MIXRT_MAX_TEX_CHANNELS);
    if (d->mode == MIXRT_DISP_SH_VEC3 && (d->sh_degree < 0 || d->sh_degree > 3))
        return vfail(m, MIXRT_EUNSUPPORTED, "disp.sh_degree=%d outside 0..3", d->sh_degree);
    if (d->dtype != MIXRT_F32 && d->dtype != MIXRT_F16 && d->dtype != MIXRT_U8)
        return vfail(m, MIXRT_EUNSUPPORTED, "disp.dtype=%d (F32, F16 or U8)", d->dtype);
    if (d->C < 0 || stored_channels(d) < disp_channels(d) || stored_channels(d) > 256)
        return vfail(m, MIXRT_EINVAL, "disp.C=%d for %d channels used", d->C, disp_channels(d));
    if (mixrt::tex_id(d->dtype, d->mode, d->sh_degree) < 0)
        return vfail(m, MIXRT_EUNSUPPORTED, "no kernel for disp dtype %d, mode %d, degree %d",
                     d->dtype, d->mode, d->sh_degree);
    if (!d->data) return vfail(m, MIXRT_EINVAL, "disp.data is NULL");
    if (!aligned16(d->data)) return vfail(m, MIXRT_EINVAL, "disp.data not 16-byte aligned");
    if (d->mode == MIXRT_DISP_SH_VEC3 && !d->scale)
        return vfail(m, MIXRT_EINVAL, "disp.scale is NULL");
    if (d->dtype == MIXRT_U8)
        for (int i = 0; i < 2; ++i)
            if (!std::isfinite(d->q_scale[i]) || !std::isfinite(d->q_offset[i]))
                return vfail(m, MIXRT_EINVAL, "disp 8-bit dequantisation not finite");
    return MIXRT_OK;
}

int check_grid(const mixrt_hash_grid *g, Msg m)
{
    if (!g) return vfail(m, MIXRT_EINVAL, "grid is NULL");
    if (g->L < 1 || g->L > MIXRT_MAX_LEVELS)
        return vfail(m, MIXRT_EUNSUPPORTED, "grid.L=%d outside 1..%d", g->L, MIXRT_MAX_LEVELS);
    if (g->log2_T < 4 || g->log2_T > 26)
        return vfail(m, MIXRT_EUNSUPPORTED, "grid.log2_T=%d outside 4..26", g->log2_T);
    if (g->F != 2 && g->F != 4) return vfail(m, MIXRT_EUNSUPPORTED, "grid.F=%d (2 or 4)", g->F);
    if (g->N_min < 1 || g->N_max < g->N_min || g->N_max > (1 << 20))
        return vfail(m, MIXRT_EINVAL, "grid N_min=%d N_max=%d", g->N_min, g->N_max);
    if (g->dtype != MIXRT_F32 && g->dtype != MIXRT_F16)
        return vfail(m, MIXRT_EUNSUPPORTED, "grid.dtype=%d (F32 or F16)", g->dtype);
    if (!g->data) return vfail(m, MIXRT_EINVAL, "grid.data is NULL");
    if (!aligned16(g->data)) return vfail(m, MIXRT_EINVAL, "grid.data not 16-byte aligned");
    return MIXRT_OK;
}

// hidden width of the kernel (an 8-wide hidden layer runs on the 16-wide
// tile, zero-padded as its weights are loaded) and hidden-layer count of a
// valid MLP
int check_mlp(const mixrt_mlp *p, int expect_in, Msg m, int *hid, int *nhid)
{
    if (!p) return vfail(m, MIXRT_EINVAL, "mlp is NULL");
    if (p->n_layers < 0 || p->n_layers > MIXRT_MAX_LAYERS)
        return vfail(m, MIXRT_EUNSUPPORTED, "mlp.n_layers=%d outside 0..%d", p->n_layers,
                     MIXRT_MAX_LAYERS);
    if (p->view_sh_dim != 0 && p->view_sh_dim != 16)
        return vfail(m, MIXRT_EUNSUPPORTED, "mlp.view_sh_dim=%d (0 or 16)", p->view_sh_dim);
    if (expect_in >= 0 && p->width[0] != expect_in)
        return vfail(m, MIXRT_EINVAL, "mlp.width[0]=%d but L*F+view_sh_dim=%d", p->width[0],
                     expect_in);
    if (p->n_layers == 0) {
        // the MLP removed: inputs summed per component (i mod 4)
        if (p->view_sh_dim != 0)
            return vfail(m, MIXRT_EINVAL, "mlp.n_layers=0 takes no view encoding");
        if (p->width[0] < 4 || p->width[0] % 4)
            return vfail(m, MIXRT_EINVAL, "mlp.n_layers=0 needs width[0] a multiple of 4");
        *hid = 0;
        *nhid = 0;
        return MIXRT_OK;
    }
    if (p->n_layers < 2)
        return vfail(m, MIXRT_EUNSUPPORTED, "mlp.n_layers=%d (0, or 2..%d)", p->n_layers,
                     MIXRT_MAX_LAYERS);
    if (p->width[p->n_layers] != 4)
        return vfail(m, MIXRT_EINVAL, "mlp output width %d (must be 4)", p->width[p->n_layers]);
    const int h = p->width[1];
    for (int i = 1; i < p->n_layers; ++i)
        if (p->width[i] != h)
            return vfail(m, MIXRT_EUNSUPPORTED, "mlp hidden widths differ (%d vs %d)", p->width[i], h);
    if (p->width[0] % 16 || (h != 8 && h != 16 && h != 32 && h != 64))
        return vfail(m, MIXRT_EUNSUPPORTED,
                     "mlp widths in=%d hidden=%d (in %%16, hidden 8/16/32/64)", p->width[0], h);
    const int hk = h < 16 ? 16 : h;
    if (!mixrt::mlp_variant_supported(p->width[0], hk, p->n_layers - 1))
        return vfail(m, MIXRT_EUNSUPPORTED, "mlp %d->%dx%d->4 not built", p->width[0], h,
                     p->n_layers - 1);
    if (!p->data) return vfail(m, MIXRT_EINVAL, "mlp.data is NULL");
    if (!aligned16(p->data)) return vfail(m, MIXRT_EINVAL, "mlp.data not 16-byte aligned");
    *hid = hk;
    *nhid = p->n_layers - 1;
    return MIXRT_OK;
}

int check_sampling(const mixrt_sampling *s, Msg m)
{
    if (!s) return vfail(m, MIXRT_EINVAL, "sampling is NULL");
    if (s->K < 1 || s->K > MIXRT_MAX_SAMPLES)
        return vfail(m, MIXRT_EUNSUPPORTED, "sampling.K=%d outside 1..%d", s->K, MIXRT_MAX_SAMPLES);
    if (!(s->delta >= 0.0f) || !std::isfinite(s->delta))
        return vfail(m, MIXRT_EINVAL, "sampling.delta=%g", s->delta);
    if (!(s->t_term >= 0.0f && s->t_term < 1.0f))
        return vfail(m, MIXRT_EINVAL, "sampling.t_term=%g outside [0,1)", s->t_term);
    return MIXRT_OK;
}

// The render kernel's texture kind: the kind specialised for the map's
// dtype and SH degree when a kernel is built for it with this grid and MLP,
// else (Eq. 2 as printed) the kind that takes the degree at run time.
int render_tex(const mixrt_disp_tex *disp, const mixrt_hash_grid *grid, const mixrt_mlp *mlp,
               int hid, int nhid)
{
    const bool tf16 = grid->dtype == MIXRT_F16;
    const int t = mixrt::tex_id(disp->dtype, disp->mode, disp->sh_degree);
    if (t >= 0 && mixrt::render_variant_supported(t, grid->F, tf16, mlp->width[0], hid, nhid))
        return t;
    if (disp->mode == MIXRT_DISP_SH_VEC3) {
        const int g = mixrt::tex_id_any_degree(disp->dtype);
        if (mixrt::render_variant_supported(g, grid->F, tf16, mlp->width[0], hid, nhid))
            return g;
    }
    return t;
}

int validate_all(const mixrt_gbuffer *gbuf, const mixrt_camera *cams, const mixrt_disp_tex *disp,
                 const mixrt_hash_grid *grid, const mixrt_mlp *mlp, const mixrt_sampling *smp,
                 Msg m, int *hid, int *nhid)
{
    int rc;
    if ((rc = check_gbuf(gbuf, cams, m))) return rc;
    if ((rc = check_disp(disp, m))) return rc;
    if ((rc = check_grid(grid, m))) return rc;
    if ((rc = check_sampling(smp, m))) return rc;
    if (!mlp) return vfail(m, MIXRT_EINVAL, "mlp is NULL");
    if ((rc = check_mlp(mlp, grid->L * grid->F + mlp->view_sh_dim, m, hid, nhid))) return rc;
    const int tex = render_tex(disp, grid, mlp, *hid, *nhid);
    if (!mixrt::render_variant_supported(tex, grid->F, grid->dtype == MIXRT_F16, mlp->width[0],
                                         *hid, *nhid))
        return vfail(m, MIXRT_EUNSUPPORTED,
                     "no render kernel for disp (dtype %d, mode %d, degree %d), grid F=%d %s, "
                     "mlp %d->%dx%d->4",
                     disp->dtype, disp->mode, disp->sh_degree, grid->F,
                     grid->dtype == MIXRT_F16 ? "f16" : "f32", mlp->width[0], *hid, *nhid);
    return MIXRT_OK;
}

// Camera constants: rotation, centre, 1 / focal length in pixels, background.
void fill_cams(mixrt::CamK *out, const mixrt_camera *cams, int views, int H)
{
    for (int v = 0; v < views; ++v) {
        const mixrt_camera &c = cams[v];
        mixrt::CamK &k = out[v];
        for (int r = 0; r < 3; ++r) {
            for (int q = 0; q < 3; ++q) k.R[3 * r + q] = c.c2w[4 * r + q];
            k.o[r] = c.c2w[4 * r + 3];
        }
        const double half = 0.5 * (double)c.fov_y_deg * 3.14159265358979323846 / 180.0;
        k.inv_f = (float)(std::tan(half) / (0.5 * (double)H));
        for (int q = 0; q < 3; ++q) k.bg[q] = c.bg[q];
    }
}

void fill_ray_params(mixrt::RayParams &rp, const mixrt_gbuffer *g, const mixrt_camera *cams,
                     const mixrt_disp_tex *d, const mixrt_sampling *s)
{
    memset(&rp, 0, sizeof rp);
    rp.g0 = (const float4 *)g->g0;
    rp.views = g->views;
    rp.W = g->W;
    rp.H = g->H;
    rp.rays = g->views * g->H * g->W;
    const bool none = d->mode == MIXRT_DISP_NONE;
    rp.tex = none ? nullptr : d->data;
    rp.tex_scale = none ? nullptr : d->scale;
    rp.tex_R = none ? 1 : d->R;
    rp.tex_V = d->mode == MIXRT_DISP_ALONG_RAY ? d->V : 0;
    rp.tex_C = none ? 1 : stored_channels(d);
    rp.tex_degree = d->mode == MIXRT_DISP_SH_VEC3 ? d->sh_degree : 0;
    for (int i = 0; i < 2; ++i) {
        rp.q_scale[i] = d->q_scale[i];
        rp.q_offset[i] = d->q_offset[i];
    }
    rp.K = s->K;
    rp.delta = s->delta;
    rp.t_term = s->t_term;
    fill_cams(rp.cams, cams, g->views, g->H);
}

void fill_grid_params(mixrt::GridParams &gp, const mixrt_hash_grid *g)
{
    memset(&gp, 0, sizeof gp);
    gp.table = g->data;
    gp.log2_T = (uint32_t)g->log2_T;
    gp.T_mask = (uint32_t)((1ull << g->log2_T) - 1);
    gp.L = g->L;
    gp.block_from = g->L;   // no block gathers unless the render launch picks some
    gp.hash_batch = 2;
    int32_t N[MIXRT_MAX_LEVELS];
    level_table(g->L, g->N_min, g->N_max, N);
    const uint64_t T = 1ull << g->log2_T;
    for (int l = 0; l < g->L; ++l) {
        gp.N[l] = (uint32_t)N[l];
        gp.Nf[l] = (float)N[l];
        gp.Ntop[l] = (float)(N[l] - 1);
        const uint64_t side = (uint64_t)N[l] + 1;
        if (side * side * side <= T) {
            gp.dense_mask |= 1u << l;
            gp.n_dense = l + 1;  // resolutions increase, so dense levels are a prefix
        }
    }
}

int finish_launch(mixrt_ctx *ctx, hipError_t e, const char *what)
{
    if (e != hipSuccess)
        return fail(ctx, MIXRT_EDEVICE, "%s: launch failed: %s", what, hipGetErrorString(e));
    if (ctx->flags & MIXRT_FLAG_SYNC_CHECK) {
        e = hipStreamSynchronize(ctx->stream);
        if (e == hipSuccess) e = hipGetLastError();
        if (e != hipSuccess)
            return fail(ctx, MIXRT_EDEVICE, "%s: device error: %s", what, hipGetErrorString(e));
    }
    return MIXRT_OK;
}

int bind_device(mixrt_ctx *ctx)
{
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess)
        return fail(ctx, MIXRT_EDEVICE, "hipSetDevice(%d): %s", ctx->device, hipGetErrorString(e));
    return MIXRT_OK;
}

}  // namespace

extern "C" {

const char *mixrt_status_string(int s)
{
    switch (s) {
    case MIXRT_OK: return "ok";
    case MIXRT_EINVAL: return "invalid argument";
    case MIXRT_ENOMEM: return "out of device memory";
    case MIXRT_EDEVICE: return "device (HIP) error";
    case MIXRT_EUNSUPPORTED: return "unsupported configuration";
    default: return "unknown status";
    }
}

int mixrt_mesh_plan(const mixrt_mesh_desc *desc, mixrt_mesh_info *info, char *msg, size_t cap)
{
    clear_err(nullptr);
    if (msg && cap) msg[0] = 0;
    mixrt::MeshGridHost g;
    char buf[512] = "";
    int rc;
    try {
        rc = mixrt::build_mesh_grid(desc, false, g, buf, sizeof buf);
    } catch (const std::bad_alloc &) {
        rc = MIXRT_ENOMEM;
        snprintf(buf, sizeof buf, "host allocation for the mesh grid failed");
    }
    if (rc) {
        if (msg && cap) snprintf(msg, cap, "%s", buf);
        return fail(nullptr, rc, "%s", buf);
    }
    if (info) {
        memset(info, 0, sizeof *info);
        for (int a = 0; a < 3; ++a) {
            info->grid_res[a] = g.n[a];
            info->lo[a] = (float)g.lo[a];
            info->hi[a] = (float)g.hi[a];
        }
        info->n_faces = desc->n_faces;
        info->n_refs = g.n_refs;
        info->device_bytes = mixrt::mesh_device_bytes(g, desc->n_faces);
    }
    return MIXRT_OK;
}

int mixrt_mesh_create(mixrt_ctx *ctx, const mixrt_mesh_desc *desc, mixrt_mesh **out)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    if (!out) return fail(ctx, MIXRT_EINVAL, "out is NULL");
    *out = nullptr;
    mixrt::MeshGridHost g;
    char buf[512] = "";
    int rc;
    try {
        // the grid's lists can reach 2^31 entries (48 bytes each) on the host
        rc = mixrt::build_mesh_grid(desc, true, g, buf, sizeof buf);
    } catch (const std::bad_alloc &) {
        return fail(ctx, MIXRT_ENOMEM, "host allocation for the mesh grid failed");
    }
    if (rc) return fail(ctx, rc, "%s", buf);
    if ((rc = bind_device(ctx))) return rc;
    const int64_t cells = (int64_t)g.n[0] * g.n[1] * g.n[2];
    const int64_t b_cells = (cells * 8 + 255) & ~int64_t(255);
    const int64_t b_refs = (g.n_refs * 48 + 255) & ~int64_t(255);
    const int64_t bytes = mixrt::mesh_device_bytes(g, desc->n_faces);
    mixrt_mesh *mesh = new (std::nothrow) mixrt_mesh;
    if (!mesh) return fail(ctx, MIXRT_ENOMEM, "host allocation failed");
    hipError_t e = hipMalloc(&mesh->mem, (size_t)bytes);
    if (e != hipSuccess) {
        delete mesh;
        return fail(ctx, MIXRT_ENOMEM, "hipMalloc(%lld) for the mesh: %s", (long long)bytes,
                    hipGetErrorString(e));
    }
    char *base = (char *)mesh->mem;
    e = hipMemcpy(base, g.cells.data(), (size_t)cells * 8, hipMemcpyHostToDevice);
    if (e == hipSuccess && g.n_refs)
        e = hipMemcpy(base + b_cells, g.refs.data(), (size_t)g.n_refs * 48, hipMemcpyHostToDevice);
    const int64_t b_attr = (desc->n_faces * 32 + 255) & ~int64_t(255);
    if (e == hipSuccess)
        e = hipMemcpy(base + b_cells + b_refs, g.attr.data(), (size_t)desc->n_faces * 32,
                      hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemcpy(base + b_cells + b_refs + b_attr, g.tris.data(), (size_t)desc->n_faces * 48,
                      hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(mesh->mem);
        delete mesh;
        return fail(ctx, MIXRT_EDEVICE, "mesh upload: %s", hipGetErrorString(e));
    }
    mesh->device = ctx->device;
    mixrt::MeshGridK &k = mesh->k;
    for (int a = 0; a < 3; ++a) {
        k.lo[a] = (float)g.lo[a];
        k.hi[a] = (float)g.hi[a];
        k.cell[a] = (float)g.cell[a];
        k.inv_cell[a] = (float)(1.0 / g.cell[a]);
        k.n[a] = g.n[a];
        mesh->info.grid_res[a] = g.n[a];
        mesh->info.lo[a] = k.lo[a];
        mesh->info.hi[a] = k.hi[a];
    }
    k.cells = (const uint2 *)base;
    k.refs = (const float4 *)(base + b_cells);
    k.attr = (const float4 *)(base + b_cells + b_refs);
    k.tris = (const float4 *)(base + b_cells + b_refs + b_attr);
    k.n_faces = (int32_t)desc->n_faces;
    mesh->info.n_faces = desc->n_faces;
    mesh->info.n_refs = g.n_refs;
    mesh->info.device_bytes = bytes;
    *out = mesh;
    return MIXRT_OK;
}

int mixrt_mesh_get_info(const mixrt_mesh *mesh, mixrt_mesh_info *info)
{
    clear_err(nullptr);
    if (!mesh || !info) return fail(nullptr, MIXRT_EINVAL, "mesh or info is NULL");
    *info = mesh->info;
    return MIXRT_OK;
}

int mixrt_mesh_destroy(mixrt_mesh *mesh)
{
    clear_err(nullptr);
    if (!mesh) return MIXRT_OK;
    int prev = 0;
    hipError_t e = hipGetDevice(&prev);
    if (e == hipSuccess) e = hipSetDevice(mesh->device);
    if (e == hipSuccess) e = hipFree(mesh->mem);
    (void)hipSetDevice(prev);
    delete mesh;
    if (e != hipSuccess) return fail(nullptr, MIXRT_EDEVICE, "mesh free: %s", hipGetErrorString(e));
    return MIXRT_OK;
}

int mixrt_raycast(mixrt_ctx *ctx, const mixrt_mesh *mesh, int32_t views, int32_t W, int32_t H,
                  const mixrt_camera *cams, float *out_g0, float *out_g1)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    if (!mesh) return fail(ctx, MIXRT_EINVAL, "mesh is NULL");
    if (mesh->device != ctx->device)
        return fail(ctx, MIXRT_EINVAL, "mesh lives on device %d, ctx on device %d", mesh->device,
                    ctx->device);
    if (views < 1 || views > MIXRT_MAX_VIEWS)
        return fail(ctx, MIXRT_EINVAL, "views=%d outside 1..%d", views, MIXRT_MAX_VIEWS);
    if (W < 1 || H < 1) return fail(ctx, MIXRT_EINVAL, "W=%d H=%d", W, H);
    if ((int64_t)views * H * W >= ((int64_t)1 << 31))
        return fail(ctx, MIXRT_EUNSUPPORTED, "more than 2^31-1 pixels per call");
    char msg[512];
    int rc = check_cams(cams, views, Msg{msg, sizeof msg});
    if (rc) return fail(ctx, rc, "%s", msg);
    if (!out_g0 || !aligned16(out_g0))
        return fail(ctx, MIXRT_EINVAL, "out_g0 is NULL or not 16-byte aligned");
    if (out_g1 && !aligned16(out_g1)) return fail(ctx, MIXRT_EINVAL, "out_g1 not 16-byte aligned");
    if ((rc = bind_device(ctx))) return rc;
    mixrt::RaycastLaunch L;
    memset(&L, 0, sizeof L);
    L.grid = mesh->k;
    fill_cams(L.cams, cams, views, H);
    L.views = views;
    L.W = W;
    L.H = H;
    L.g0 = (float4 *)out_g0;
    L.g1 = (float4 *)out_g1;
    return finish_launch(ctx, mixrt::launch_raycast(L, ctx->stream), "raycast");
}

int mixrt_rasterize(mixrt_ctx *ctx, const mixrt_mesh *mesh, int32_t views, int32_t W, int32_t H,
                    const mixrt_camera *cams, float *out_g0, float *out_g1)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    if (!mesh) return fail(ctx, MIXRT_EINVAL, "mesh is NULL");
    if (mesh->device != ctx->device)
        return fail(ctx, MIXRT_EINVAL, "mesh lives on device %d, ctx on device %d", mesh->device,
                    ctx->device);
    if (views < 1 || views > MIXRT_MAX_VIEWS)
        return fail(ctx, MIXRT_EINVAL, "views=%d outside 1..%d", views, MIXRT_MAX_VIEWS);
    if (W < 1 || H < 1) return fail(ctx, MIXRT_EINVAL, "W=%d H=%d", W, H);
    if ((int64_t)W * H >= ((int64_t)1 << 26) || (int64_t)views * H * W >= ((int64_t)1 << 31))
        return fail(ctx, MIXRT_EUNSUPPORTED, "rasterize takes fewer than 2^26 pixels per view");
    char msg[512];
    int rc = check_cams(cams, views, Msg{msg, sizeof msg});
    if (rc) return fail(ctx, rc, "%s", msg);
    if (!out_g0 || !aligned16(out_g0))
        return fail(ctx, MIXRT_EINVAL, "out_g0 is NULL or not 16-byte aligned");
    if (out_g1 && !aligned16(out_g1)) return fail(ctx, MIXRT_EINVAL, "out_g1 not 16-byte aligned");
    if ((rc = bind_device(ctx))) return rc;
    mixrt::RasterLaunch L;
    memset(&L, 0, sizeof L);
    L.tris = mesh->k.tris;
    L.attr = mesh->k.attr;
    L.n_faces = mesh->k.n_faces;
    fill_cams(L.cams, cams, views, H);
    for (int v = 0; v < views; ++v) {
        // Clip depth: half of t_min times the smallest |d_z| of the view's
        // pixel rays (reached at a corner), so every hit with t > t_min lies
        // in front of the clipping plane.
        const double inv_f = L.cams[v].inv_f;
        const double cx = (0.5 * W) * inv_f, cy = (0.5 * H) * inv_f;
        const double dz = 1.0 / std::sqrt(cx * cx + cy * cy + 1.0);
        L.near_z[v] = (float)(0.5 * (double)MIXRT_RAY_T_MIN * dz);
    }
    L.views = views;
    L.W = W;
    L.H = H;
    L.g0 = (float4 *)out_g0;
    L.g1 = (float4 *)out_g1;
    return finish_launch(ctx, mixrt::launch_rasterize(L, ctx->stream), "rasterize");
}

const char *mixrt_last_error(const mixrt_ctx *ctx) { return ctx ? ctx->err.c_str() : ""; }

const char *mixrt_thread_error(void) { return t_err.c_str(); }

int mixrt_validate(const mixrt_gbuffer *gbuf, const mixrt_camera *cams, const mixrt_disp_tex *disp,
                   const mixrt_hash_grid *grid, const mixrt_mlp *mlp, const mixrt_sampling *smp,
                   char *msg, size_t cap)
{
    if (msg && cap) msg[0] = 0;
    int hid = 0, nhid = 0;
    return validate_all(gbuf, cams, disp, grid, mlp, smp, Msg{msg, cap}, &hid, &nhid);
}

int mixrt_level_resolutions(const mixrt_hash_grid *grid, int32_t *out_N)
{
    char buf[256];
    if (!out_N) return fail(nullptr, MIXRT_EINVAL, "out_N is NULL");
    if (!grid) return fail(nullptr, MIXRT_EINVAL, "grid is NULL");
    if (grid->L < 1 || grid->L > MIXRT_MAX_LEVELS || grid->N_min < 1 || grid->N_max < grid->N_min ||
        grid->N_max > (1 << 20)) {
        snprintf(buf, sizeof buf, "grid L=%d N_min=%d N_max=%d", grid->L, grid->N_min, grid->N_max);
        return fail(nullptr, MIXRT_EINVAL, "%s", buf);
    }
    level_table(grid->L, grid->N_min, grid->N_max, out_N);
    return MIXRT_OK;
}

int mixrt_create(mixrt_ctx **out, const mixrt_create_info *ci)
{
    clear_err(nullptr);
    if (!out) return fail(nullptr, MIXRT_EINVAL, "out is NULL");
    *out = nullptr;
    if (!ci) return fail(nullptr, MIXRT_EINVAL, "create_info is NULL");
    constexpr uint32_t known = MIXRT_FLAG_SYNC_CHECK | MIXRT_FLAG_BLOCKS_FULL | MIXRT_FLAG_BLOCKS_TWO;
    if (ci->flags & ~known)
        return fail(nullptr, MIXRT_EINVAL, "unknown flags 0x%x", ci->flags & ~known);
    if ((ci->flags & MIXRT_FLAG_BLOCKS_FULL) && (ci->flags & MIXRT_FLAG_BLOCKS_TWO))
        return fail(nullptr, MIXRT_EINVAL, "MIXRT_FLAG_BLOCKS_FULL and MIXRT_FLAG_BLOCKS_TWO together");
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess || n == 0)
        return fail(nullptr, MIXRT_EDEVICE, "no HIP device: %s", hipGetErrorString(e));
    if (ci->device < 0 || ci->device >= n)
        return fail(nullptr, MIXRT_EINVAL, "device %d outside 0..%d", ci->device, n - 1);
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, ci->device);
    if (e != hipSuccess)
        return fail(nullptr, MIXRT_EDEVICE, "hipGetDeviceProperties: %s", hipGetErrorString(e));
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(nullptr, MIXRT_EUNSUPPORTED, "device %d is %s, this library is built for gfx950",
                    ci->device, prop.gcnArchName);
    // the render kernels' work counters: one small zeroed buffer per
    // context, allocated on its device (the caller's current device is kept)
    int prev = 0;
    if ((e = hipGetDevice(&prev)) != hipSuccess || (e = hipSetDevice(ci->device)) != hipSuccess)
        return fail(nullptr, MIXRT_EDEVICE, "hipSetDevice(%d): %s", ci->device, hipGetErrorString(e));
    unsigned int *work = nullptr;
    e = hipMalloc((void **)&work, mixrt::kWorkWords * sizeof(unsigned int));
    if (e == hipSuccess) e = hipMemset(work, 0, mixrt::kWorkWords * sizeof(unsigned int));
    // (done before any stream of the caller's can launch a render on it)
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        if (work) (void)hipFree(work);
        (void)hipSetDevice(prev);
        return fail(nullptr, e == hipErrorOutOfMemory ? MIXRT_ENOMEM : MIXRT_EDEVICE,
                    "work counters: %s", hipGetErrorString(e));
    }
    // and, once per device, the no-alloc render's counters
    e = scratch_setup(ci->device);
    if (e != hipSuccess) {
        (void)hipFree(work);
        (void)hipSetDevice(prev);
        return fail(nullptr, MIXRT_EDEVICE, "no-alloc work counters: %s", hipGetErrorString(e));
    }
    (void)hipSetDevice(prev);
    mixrt_ctx *ctx = new (std::nothrow) mixrt_ctx;
    if (!ctx) {
        (void)hipFree(work);
        return fail(nullptr, MIXRT_ENOMEM, "host allocation failed");
    }
    ctx->work = work;
    ctx->device = ci->device;
    ctx->stream = (hipStream_t)ci->hip_stream;
    ctx->flags = ci->flags;
    ctx->tile_stripe = ci->tile_stripe;
    ctx->early_stop_chunk = ci->early_stop_chunk;
    ctx->block_levels = ci->block_levels;
    ctx->cus = prop.multiProcessorCount;
    ctx->l2_bytes = prop.l2CacheSize;
    *out = ctx;
    return MIXRT_OK;
}

int mixrt_destroy(mixrt_ctx *ctx)
{
    if (!ctx) return MIXRT_OK;
    if (ctx->work) {
        // freed once the context's stream has finished the work enqueued on it
        int prev = 0;
        if (hipGetDevice(&prev) == hipSuccess && hipSetDevice(ctx->device) == hipSuccess) {
            (void)hipStreamSynchronize(ctx->stream);
            (void)hipFree(ctx->work);
            (void)hipSetDevice(prev);
        }
    }
    delete ctx;
    return MIXRT_OK;
}

int mixrt_sync(mixrt_ctx *ctx)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    int rc = bind_device(ctx);
    if (rc) return rc;
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess)
        return fail(ctx, MIXRT_EDEVICE, "stream synchronize: %s", hipGetErrorString(e));
    return MIXRT_OK;
}

namespace {

// The launch of a render call whose descriptors validated (hid, nhid: the
// MLP's hidden width and hidden-layer count).
void fill_render_launch(mixrt::RenderLaunch &L, const mixrt_ctx *ctx, const mixrt_gbuffer *gbuf,
                        const mixrt_camera *cams, const mixrt_disp_tex *disp,
                        const mixrt_hash_grid *grid, const mixrt_mlp *mlp,
                        const mixrt_sampling *smp, int hid, int nhid, float *out_rgba)
{
    fill_ray_params(L.rp, gbuf, cams, disp, smp);
    fill_grid_params(L.gp, grid);
    L.weights = (const _Float16 *)mlp->data;
    L.out = (float4 *)out_rgba;
    L.view_sh = mlp->view_sh_dim;
    L.tex = render_tex(disp, grid, mlp, hid, nhid);
    L.tf16 = grid->dtype == MIXRT_F16;
    L.F = grid->F;
    L.in = mlp->width[0];
    L.hid = hid;
    L.nhid = nhid;
    L.hid_w = nhid > 0 ? mlp->width[1] : 0;
    L.cus = ctx->cus;
    L.l2_bytes = ctx->l2_bytes;
    L.blocks_mode = (ctx->flags & MIXRT_FLAG_BLOCKS_FULL) ? 1 : (ctx->flags & MIXRT_FLAG_BLOCKS_TWO) ? 2 : 0;
    L.tile_stripe = ctx->tile_stripe;
    L.chunk = ctx->early_stop_chunk;
    L.block_levels = ctx->block_levels;
    L.work = ctx->work;
}

}  // namespace

namespace {

// mixrt_render with the kernels' work counters at `work` (null: the
// context's own)
int render_with(mixrt_ctx *ctx, const mixrt_gbuffer *gbuf, const mixrt_camera *cams,
                const mixrt_disp_tex *disp, const mixrt_hash_grid *grid, const mixrt_mlp *mlp,
                const mixrt_sampling *smp, float *out_rgba, bool noalloc)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    char msg[512];
    int hid = 0, nhid = 0;
    int rc = validate_all(gbuf, cams, disp, grid, mlp, smp, Msg{msg, sizeof msg}, &hid, &nhid);
    if (rc) return fail(ctx, rc, "%s", msg);
    if (!out_rgba) return fail(ctx, MIXRT_EINVAL, "out_rgba is NULL");
    if (!aligned16(out_rgba)) return fail(ctx, MIXRT_EINVAL, "out_rgba not 16-byte aligned");
    unsigned int *work = ctx->work;
    if (noalloc) {
        work = ctx->device < kMaxScratchDevices ? g_scratch[ctx->device].load() : nullptr;
        if (!work)
            return fail(ctx, MIXRT_EUNSUPPORTED, "no no-alloc work counters on device %d",
                        ctx->device);
    }
    if ((rc = bind_device(ctx))) return rc;
    mixrt::RenderLaunch L;
    fill_render_launch(L, ctx, gbuf, cams, disp, grid, mlp, smp, hid, nhid, out_rgba);
    L.work = work;
    return finish_launch(ctx, mixrt::launch_render(L, ctx->stream), noalloc ? "render_noalloc" : "render");
}

}  // namespace

int mixrt_render(mixrt_ctx *ctx, const mixrt_gbuffer *gbuf, const mixrt_camera *cams,
                 const mixrt_disp_tex *disp, const mixrt_hash_grid *grid, const mixrt_mlp *mlp,
                 const mixrt_sampling *smp, float *out_rgba)
{
    return render_with(ctx, gbuf, cams, disp, grid, mlp, smp, out_rgba, false);
}

int mixrt_render_noalloc(mixrt_ctx *ctx, const mixrt_gbuffer *gbuf, const mixrt_camera *cams,
                         const mixrt_disp_tex *disp, const mixrt_hash_grid *grid,
                         const mixrt_mlp *mlp, const mixrt_sampling *smp, float *out_rgba)
{
    return render_with(ctx, gbuf, cams, disp, grid, mlp, smp, out_rgba, true);
}

int mixrt_render_launch_shape(mixrt_ctx *ctx, const mixrt_gbuffer *gbuf,
                              const mixrt_camera *cams, const mixrt_disp_tex *disp,
                              const mixrt_hash_grid *grid, const mixrt_mlp *mlp,
                              const mixrt_sampling *smp, mixrt_launch_plan *plan)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    char msg[512];
    int hid = 0, nhid = 0;
    int rc = validate_all(gbuf, cams, disp, grid, mlp, smp, Msg{msg, sizeof msg}, &hid, &nhid);
    if (rc) return fail(ctx, rc, "%s", msg);
    if (!plan) return fail(ctx, MIXRT_EINVAL, "plan is NULL");
    if ((rc = bind_device(ctx))) return rc;
    mixrt::RenderLaunch L;
    fill_render_launch(L, ctx, gbuf, cams, disp, grid, mlp, smp, hid, nhid, nullptr);
    int b = 0, st = 0, ch = 0, bf = 0, hb = 0, cl = 0;
    const hipError_t e = mixrt::render_launch_shape(L, &b, &st, &ch, &bf, &hb, &cl);
    if (e != hipSuccess)
        return fail(ctx, MIXRT_EDEVICE, "render launch shape: %s", hipGetErrorString(e));
    plan->blocks = b;
    plan->tile_stripe = st;
    plan->chunk = ch;
    plan->block_from = bf;
    plan->hash_batch = hb;
    plan->claims = cl;
    return MIXRT_OK;
}

int mixrt_debug_phase_cycles(mixrt_ctx *ctx, uint64_t *out, int reset)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    if (!out) return fail(ctx, MIXRT_EINVAL, "out is NULL");
    int rc = bind_device(ctx);
    if (rc) return rc;
    const hipError_t e = mixrt::phase_cycles_read(out, reset != 0);
    if (e == hipErrorNotSupported)
        return fail(ctx, MIXRT_EUNSUPPORTED, "this library is not the phase-timer build");
    if (e != hipSuccess) return fail(ctx, MIXRT_EDEVICE, "phase cycles: %s", hipGetErrorString(e));
    return MIXRT_OK;
}

int mixrt_debug_ray_setup(mixrt_ctx *ctx, const mixrt_gbuffer *gbuf, const mixrt_camera *cams,
                          const mixrt_disp_tex *disp, const mixrt_sampling *smp, float *out_x,
                          int32_t *out_hit)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    char msg[512];
    Msg m{msg, sizeof msg};
    int rc;
    if ((rc = check_gbuf(gbuf, cams, m)) || (rc = check_disp(disp, m)) ||
        (rc = check_sampling(smp, m)))
        return fail(ctx, rc, "%s", msg);
    if (!out_x) return fail(ctx, MIXRT_EINVAL, "out_x is NULL");
    if ((rc = bind_device(ctx))) return rc;
    mixrt::RayParams rp;
    fill_ray_params(rp, gbuf, cams, disp, smp);
    return finish_launch(ctx,
                         mixrt::launch_ray_setup(
                             rp, mixrt::tex_id(disp->dtype, disp->mode, disp->sh_degree), out_x,
                             out_hit, ctx->stream),
                         "ray_setup");
}

int mixrt_debug_hash_encode(mixrt_ctx *ctx, const mixrt_hash_grid *grid, const float *x, int64_t n,
                            int32_t *out_corner, uint32_t *out_idx, float *out_w, float *out_feat)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    char msg[512];
    int rc = check_grid(grid, Msg{msg, sizeof msg});
    if (rc) return fail(ctx, rc, "%s", msg);
    if (n < 0 || n >= ((int64_t)1 << 31)) return fail(ctx, MIXRT_EINVAL, "n=%lld", (long long)n);
    if (n > 0 && !x) return fail(ctx, MIXRT_EINVAL, "x is NULL");
    if ((rc = bind_device(ctx))) return rc;
    mixrt::GridParams gp;
    fill_grid_params(gp, grid);
    return finish_launch(ctx,
                         mixrt::launch_hash_encode(gp, grid->F, grid->dtype == MIXRT_F16, x, n,
                                                   out_corner, out_idx, out_w, out_feat,
                                                   ctx->stream),
                         "hash_encode");
}

int mixrt_debug_mlp(mixrt_ctx *ctx, const mixrt_mlp *mlp, const uint16_t *in_f16, int64_t n,
                    float *out4)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    char msg[512];
    int hid = 0, nhid = 0;
    int rc = check_mlp(mlp, -1, Msg{msg, sizeof msg}, &hid, &nhid);
    if (rc) return fail(ctx, rc, "%s", msg);
    if (n < 0 || n >= ((int64_t)1 << 40)) return fail(ctx, MIXRT_EINVAL, "n=%lld", (long long)n);
    if (n > 0 && (!in_f16 || !out4)) return fail(ctx, MIXRT_EINVAL, "in or out is NULL");
    if (n > 0 && (!aligned16(in_f16) || !aligned16(out4)))
        return fail(ctx, MIXRT_EINVAL, "in_f16/out4 not 16-byte aligned");
    if ((rc = bind_device(ctx))) return rc;
    return finish_launch(ctx,
                         mixrt::launch_mlp(mlp->width[0], hid, nhid,
                                           nhid > 0 ? mlp->width[1] : 0,
                                           (const _Float16 *)mlp->data, (const _Float16 *)in_f16,
                                           n, (float4 *)out4, ctx->cus, ctx->stream),
                         "mlp");
}

int mixrt_debug_composite(mixrt_ctx *ctx, const float *srgb, int64_t rays,
                          const mixrt_sampling *smp, const float *bg, float *out_rgba)
{
    if (!ctx) return fail(nullptr, MIXRT_EINVAL, "ctx is NULL");
    clear_err(ctx);
    char msg[512];
    int rc = check_sampling(smp, Msg{msg, sizeof msg});
    if (rc) return fail(ctx, rc, "%s", msg);
    if (!bg) return fail(ctx, MIXRT_EINVAL, "bg is NULL");
    if (rays < 0) return fail(ctx, MIXRT_EINVAL, "rays=%lld", (long long)rays);
    if (rays > 0 && (!srgb || !out_rgba)) return fail(ctx, MIXRT_EINVAL, "srgb or out is NULL");
    if (rays > 0 && (!aligned16(srgb) || !aligned16(out_rgba)))
        return fail(ctx, MIXRT_EINVAL, "srgb/out_rgba not 16-byte aligned");
    if ((rc = bind_device(ctx))) return rc;
    return finish_launch(ctx,
                         mixrt::launch_composite((const float4 *)srgb, rays, smp->K, smp->delta,
                                                 smp->t_term, bg, (float4 *)out_rgba, ctx->stream),
                         "composite");
}

}  // extern "C"
