// Internal interface of the geometry stage, which produces the G-buffer of
// the coarse mesh (Fig. 2 step 1): the uploaded mesh (triangle records and the
// uniform grid of triangle lists, built on the host in mixrt_mesh.cpp), the
// rasteriser (mixrt_raster.hip) and the ray-casting kernel that walks the grid
// (mixrt_raycast.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "mixrt.h"
#include "mixrt_device.hpp"

namespace mixrt {

inline constexpr int kMaxGridAxis = 1024;
inline constexpr int64_t kMaxGridCells = int64_t(1) << 26;
// Triangle boxes are padded by this fraction of a cell when binned, so that
// a hit computed in fp32 near a cell face is listed in the cell on either side.
inline constexpr double kBinPad = 1.0 / 500.0;

// Device view of an uploaded mesh.  Cell (x, y, z) is index (z*ny + y)*nx + x
// and cells[c] = (first, count): a cell with triangles lists them in
// refs[first .. first+count); an empty cell (count 0) holds in `first` its
// Chebyshev distance D (in cells, 1..255) to the nearest cell with
// triangles, so every cell within D-1 of it on each axis is empty as well.
// A ref is three float4: (v0, triangle index bits), (e1, 0), (e2, 0).
// attr[tri] is two float4: (uv0, uv1), (uv2, 0, 0).
struct MeshGridK {
    float lo[3], hi[3], cell[3], inv_cell[3];
    int32_t n[3];
    const uint2 *cells;
    const float4 *refs;
    const float4 *attr;
    const float4 *tris;   // [n_faces] records like refs, in triangle order
    int32_t n_faces;
};

// The grid as built on the host, before upload.
struct MeshGridHost {
    int32_t n[3] = {0, 0, 0};
    double lo[3] = {0, 0, 0}, hi[3] = {0, 0, 0}, cell[3] = {0, 0, 0};
    int64_t n_refs = 0;
    std::vector<uint32_t> cells;        // 2 per cell: (first or distance, count)
    std::vector<float> refs;            // n_refs * 12
    std::vector<float> attr;            // n_faces * 8
    std::vector<float> tris;            // n_faces * 12, triangle order
};

// Validate desc and choose bounds and resolution; with fill, also count and
// fill the cell lists (otherwise only n_refs is computed).  Returns a
// mixrt_status and writes a message to msg on failure.
int build_mesh_grid(const mixrt_mesh_desc *desc, bool fill, MeshGridHost &g, char *msg,
                    size_t cap);

// Bytes of device memory an uploaded grid occupies (each array 256-aligned).
int64_t mesh_device_bytes(const MeshGridHost &g, int64_t n_faces);

struct RaycastLaunch {
    MeshGridK grid;
    CamK cams[MIXRT_MAX_VIEWS];
    int32_t views, W, H;
    float4 *g0;
    float4 *g1;
};

hipError_t launch_raycast(const RaycastLaunch &L, hipStream_t stream);

// The rasteriser: per view, triangles are clipped at camera depth near_z
// (chosen on the host so that no hit with t > MIXRT_RAY_T_MIN is closer).
// Pixels per view must be below 2^26 (box areas of a wave sum in 32 bits).
struct RasterLaunch {
    const float4 *tris;
    const float4 *attr;
    int32_t n_faces;
    CamK cams[MIXRT_MAX_VIEWS];
    float near_z[MIXRT_MAX_VIEWS];
    int32_t views, W, H;
    float4 *g0;
    float4 *g1;
};

hipError_t launch_rasterize(const RasterLaunch &L, hipStream_t stream);

}  // namespace mixrt
