// Host-side construction of a mesh's device arrays: the uniform grid of
// triangle lists that the ray-casting kernel walks (mixrt_raycast.hip) and the
// triangle records the rasteriser reads (mixrt_raster.hip).  Deterministic: the result
// depends only on the descriptor, and every cell lists its triangles in
// ascending index order.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>

#include "mixrt_mesh.hpp"

namespace mixrt {

namespace {

int msgf(char *msg, size_t cap, int code, const char *fmt, ...)
{
    if (msg && cap) {
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(msg, cap, fmt, ap);
        va_end(ap);
    }
    return code;
}

int64_t align256(int64_t b) { return (b + 255) & ~int64_t(255); }

// Inclusive cell range of [a, b] on one axis, clamped to the grid.
void cell_range(const MeshGridHost &g, int axis, double a, double b, int &c0, int &c1)
{
    const double inv = g.n[axis] / (g.hi[axis] - g.lo[axis]);
    const double pad = kBinPad * g.cell[axis];
    c0 = (int)floor((a - pad - g.lo[axis]) * inv);
    c1 = (int)floor((b + pad - g.lo[axis]) * inv);
    c0 = std::min(std::max(c0, 0), g.n[axis] - 1);
    c1 = std::min(std::max(c1, 0), g.n[axis] - 1);
}

// Visit every cell whose padded box the triangle's plane crosses, within the
// triangle's padded bounding box.
template <class F>
void for_cells(const MeshGridHost &g, const double p[3][3], F &&visit)
{
    int lo[3], hi[3];
    for (int a = 0; a < 3; ++a) {
        const double mn = std::min(p[0][a], std::min(p[1][a], p[2][a]));
        const double mx = std::max(p[0][a], std::max(p[1][a], p[2][a]));
        cell_range(g, a, mn, mx, lo[a], hi[a]);
    }
    double e1[3], e2[3];
    for (int a = 0; a < 3; ++a) {
        e1[a] = p[1][a] - p[0][a];
        e2[a] = p[2][a] - p[0][a];
    }
    const double nrm[3] = {e1[1] * e2[2] - e1[2] * e2[1], e1[2] * e2[0] - e1[0] * e2[2],
                           e1[0] * e2[1] - e1[1] * e2[0]};
    const bool single = lo[0] == hi[0] && lo[1] == hi[1] && lo[2] == hi[2];
    double half[3];
    for (int a = 0; a < 3; ++a) half[a] = g.cell[a] * (0.5 + kBinPad);
    const double reach = fabs(nrm[0]) * half[0] + fabs(nrm[1]) * half[1] + fabs(nrm[2]) * half[2];
    const int64_t nx = g.n[0], ny = g.n[1];
    for (int z = lo[2]; z <= hi[2]; ++z)
        for (int y = lo[1]; y <= hi[1]; ++y)
            for (int x = lo[0]; x <= hi[0]; ++x) {
                if (!single) {
                    const double c[3] = {g.lo[0] + (x + 0.5) * g.cell[0],
                                         g.lo[1] + (y + 0.5) * g.cell[1],
                                         g.lo[2] + (z + 0.5) * g.cell[2]};
                    const double dist = nrm[0] * (c[0] - p[0][0]) + nrm[1] * (c[1] - p[0][1]) +
                                        nrm[2] * (c[2] - p[0][2]);
                    if (fabs(dist) > reach * (1.0 + 1e-9)) continue;
                }
                visit(((int64_t)z * ny + y) * nx + x);
            }
}

// Chebyshev distance transform of the occupancy: dist 0 on cells with
// triangles, else the largest D (capped at 255) such that every cell within
// D-1 on each axis is empty.  Two raster passes with the 26-neighbourhood
// give the exact chessboard distance; cells beyond the grid count as empty.
void chessboard_distance(const int32_t n[3], std::vector<uint8_t> &dist)
{
    const int nx = n[0], ny = n[1], nz = n[2];
    auto at = [&](int x, int y, int z) -> uint8_t & {
        return dist[((int64_t)z * ny + y) * nx + x];
    };
    for (int pass = 0; pass < 2; ++pass) {
        const int s = pass == 0 ? 1 : -1;
        for (int zi = 0; zi < nz; ++zi)
            for (int yi = 0; yi < ny; ++yi)
                for (int xi = 0; xi < nx; ++xi) {
                    const int x = pass == 0 ? xi : nx - 1 - xi;
                    const int y = pass == 0 ? yi : ny - 1 - yi;
                    const int z = pass == 0 ? zi : nz - 1 - zi;
                    uint8_t &d = at(x, y, z);
                    if (d == 0) continue;
                    int best = d;
                    // the 13 neighbours already visited in this pass's order
                    for (int dz = -1; dz <= 0; ++dz)
                        for (int dy = -1; dy <= 1; ++dy)
                            for (int dx = -1; dx <= 1; ++dx) {
                                if (dz == 0 && (dy > 0 || (dy == 0 && dx >= 0))) continue;
                                const int X = x + s * dx, Y = y + s * dy, Z = z + s * dz;
                                if (X < 0 || Y < 0 || Z < 0 || X >= nx || Y >= ny || Z >= nz)
                                    continue;
                                best = std::min(best, at(X, Y, Z) + 1);
                            }
                    d = (uint8_t)std::min(best, 255);
                }
    }
}

void load_tri(const mixrt_mesh_desc *d, int64_t f, double p[3][3])
{
    for (int k = 0; k < 3; ++k) {
        const int64_t v = d->faces[3 * f + k];
        for (int a = 0; a < 3; ++a) p[k][a] = d->positions[3 * v + a];
    }
}

}  // namespace

int64_t mesh_device_bytes(const MeshGridHost &g, int64_t n_faces)
{
    const int64_t cells = (int64_t)g.n[0] * g.n[1] * g.n[2];
    return align256(cells * 8) + align256(g.n_refs * 48) + align256(n_faces * 32) +
           align256(n_faces * 48);
}

int build_mesh_grid(const mixrt_mesh_desc *d, bool fill, MeshGridHost &g, char *msg, size_t cap)
{
    g = MeshGridHost();
    if (!d) return msgf(msg, cap, MIXRT_EINVAL, "mesh desc is NULL");
    const int64_t lim = (int64_t(1) << 31) - 1;
    if (d->n_vertices < 3 || d->n_vertices > lim)
        return msgf(msg, cap, MIXRT_EINVAL, "mesh n_vertices=%lld", (long long)d->n_vertices);
    if (d->n_faces < 1 || d->n_faces > lim)
        return msgf(msg, cap, MIXRT_EINVAL, "mesh n_faces=%lld", (long long)d->n_faces);
    if (!d->positions || !d->faces)
        return msgf(msg, cap, MIXRT_EINVAL, "mesh positions or faces is NULL");
    const bool autores = d->grid_res[0] == 0 && d->grid_res[1] == 0 && d->grid_res[2] == 0;
    if (!autores) {
        int64_t cells = 1;
        for (int a = 0; a < 3; ++a) {
            if (d->grid_res[a] < 1 || d->grid_res[a] > kMaxGridAxis)
                return msgf(msg, cap, MIXRT_EINVAL, "mesh grid_res[%d]=%d outside 1..%d", a,
                            d->grid_res[a], kMaxGridAxis);
            cells *= d->grid_res[a];
        }
        if (cells > kMaxGridCells)
            return msgf(msg, cap, MIXRT_EINVAL, "mesh grid of %lld cells (at most 2^26)",
                        (long long)cells);
    }
    if (!(d->cells_per_face >= 0.0f && d->cells_per_face <= 64.0f))
        return msgf(msg, cap, MIXRT_EINVAL, "mesh cells_per_face=%g outside [0, 64]",
                    (double)d->cells_per_face);
    for (int64_t i = 0; i < 3 * d->n_faces; ++i)
        if (d->faces[i] < 0 || d->faces[i] >= d->n_vertices)
            return msgf(msg, cap, MIXRT_EINVAL, "mesh face %lld has vertex index %d",
                        (long long)(i / 3), d->faces[i]);
    double lo[3] = {INFINITY, INFINITY, INFINITY}, hi[3] = {-INFINITY, -INFINITY, -INFINITY};
    for (int64_t v = 0; v < d->n_vertices; ++v)
        for (int a = 0; a < 3; ++a) {
            const double x = d->positions[3 * v + a];
            if (!isfinite(x))
                return msgf(msg, cap, MIXRT_EINVAL, "mesh vertex %lld is not finite", (long long)v);
            lo[a] = std::min(lo[a], x);
            hi[a] = std::max(hi[a], x);
        }
    if (d->uv)
        for (int64_t i = 0; i < 2 * d->n_vertices; ++i)
            if (!isfinite(d->uv[i]))
                return msgf(msg, cap, MIXRT_EINVAL, "mesh uv of vertex %lld is not finite",
                            (long long)(i / 2));

    // Bounds padded by 1/1000 of the largest extent (a flat mesh still gets
    // a box of positive volume), kept representable in fp32.
    double ext_max = 0.0;
    for (int a = 0; a < 3; ++a) ext_max = std::max(ext_max, hi[a] - lo[a]);
    const double pad = 1e-3 * ext_max + 1e-6 * (1.0 + std::max(fabs(lo[0]), fabs(hi[0])));
    double ext[3];
    for (int a = 0; a < 3; ++a) {
        g.lo[a] = (double)(float)(lo[a] - pad);
        ext[a] = (double)(float)(hi[a] + pad) - g.lo[a];
    }
    if (autores) {
        const double cpf = d->cells_per_face > 0.0f ? d->cells_per_face : 8.0;
        double s = cbrt(cpf * (double)d->n_faces / (ext[0] * ext[1] * ext[2]));
        for (;;) {
            int64_t cells = 1;
            for (int a = 0; a < 3; ++a) {
                g.n[a] = (int)std::min<double>(std::max(1.0, floor(ext[a] * s + 0.5)), kMaxGridAxis);
                cells *= g.n[a];
            }
            if (cells <= kMaxGridCells) break;
            s *= 0.95;
        }
    } else {
        for (int a = 0; a < 3; ++a) g.n[a] = d->grid_res[a];
    }
    for (int a = 0; a < 3; ++a) {
        g.cell[a] = (double)(float)(ext[a] / g.n[a]);
        g.hi[a] = (double)(float)(g.lo[a] + g.cell[a] * g.n[a]);
        g.cell[a] = (g.hi[a] - g.lo[a]) / g.n[a];
    }

    const int64_t cells = (int64_t)g.n[0] * g.n[1] * g.n[2];
    std::vector<uint32_t> count(fill ? cells : 0, 0);
    int64_t refs = 0;
    double p[3][3];
    for (int64_t f = 0; f < d->n_faces; ++f) {
        load_tri(d, f, p);
        for_cells(g, p, [&](int64_t c) {
            ++refs;
            if (fill) ++count[c];
        });
        if (refs >= (int64_t(1) << 31))
            return msgf(msg, cap, MIXRT_EUNSUPPORTED,
                        "mesh grid needs 2^31 or more triangle entries: use a coarser grid");
    }
    g.n_refs = refs;
    if (!fill) return MIXRT_OK;

    std::vector<uint32_t> cursor(cells);
    std::vector<uint8_t> dist(cells);
    uint32_t first = 0;
    for (int64_t c = 0; c < cells; ++c) {
        cursor[c] = first;
        first += count[c];
        dist[c] = count[c] ? 0 : 255;
    }
    chessboard_distance(g.n, dist);
    g.cells.assign(2 * cells, 0);
    for (int64_t c = 0; c < cells; ++c) {
        g.cells[2 * c] = count[c] ? cursor[c] : dist[c];
        g.cells[2 * c + 1] = count[c];
    }
    g.refs.assign(refs * 12, 0.0f);
    g.tris.assign(d->n_faces * 12, 0.0f);
    for (int64_t f = 0; f < d->n_faces; ++f) {
        load_tri(d, f, p);
        const float *v0 = d->positions + 3 * (int64_t)d->faces[3 * f];
        const float *v1 = d->positions + 3 * (int64_t)d->faces[3 * f + 1];
        const float *v2 = d->positions + 3 * (int64_t)d->faces[3 * f + 2];
        float rec[12];
        const int32_t id = (int32_t)f;
        for (int a = 0; a < 3; ++a) {
            rec[a] = v0[a];
            rec[4 + a] = v1[a] - v0[a];
            rec[8 + a] = v2[a] - v0[a];
        }
        memcpy(&rec[3], &id, 4);
        rec[7] = rec[11] = 0.0f;
        for_cells(g, p, [&](int64_t c) { memcpy(&g.refs[12 * (int64_t)cursor[c]++], rec, sizeof rec); });
        memcpy(&g.tris[12 * f], rec, sizeof rec);
    }
    g.attr.assign(d->n_faces * 8, 0.0f);
    if (d->uv)
        for (int64_t f = 0; f < d->n_faces; ++f)
            for (int k = 0; k < 3; ++k)
                for (int a = 0; a < 2; ++a)
                    g.attr[8 * f + 2 * k + a] = d->uv[2 * (int64_t)d->faces[3 * f + k] + a];
    return MIXRT_OK;
}

}  // namespace mixrt
