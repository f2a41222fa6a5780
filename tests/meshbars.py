"""Error bars of the ray-mesh hit (the geometry stage) that the GPU tests
apply to pixels the oracle calls unambiguous, shared with the CPU test that
pins them (tests/test_geometry_bars.py).

The kernels solve Moller-Trumbore in fp32 from the fp32 pixel ray and the
triangle's fp32 edges.  The ray direction's relative error (a few ulps) moves
the hit by about t * ulp / |cos| (cos between the ray and the normal); the
solve forms t from products of vectors of length about D (the farthest
vertex's distance from the camera), so it adds a few ulps of D times the
condition number S / |cos|, S = L_max^2 / (2 area) (about 1 / sin of the
smallest corner angle).  The coefficients below sit 6-7x above the largest
error of an fp32 emulation of the kernels' solve over the seeded random
soups, which the CPU test checks."""
import numpy as np

T_REL, T_COND = 2e-6, 2e-7          # t bar: (T_REL t + T_COND D S) / |cos|
UV_REL, UV_COND, UV_ABS = 1e-5, 1e-7, 1e-6


def conditioning(positions, faces, tri, origin):
    """(D, L_max, S) of triangles `tri` seen from `origin` [n, 3]."""
    P = np.asarray(positions, np.float64)[np.asarray(faces)[tri]]         # [n, 3, 3]
    dist = np.linalg.norm(P - np.asarray(origin, np.float64)[:, None, :], axis=2).max(1)
    edges = np.stack([P[:, 1] - P[:, 0], P[:, 2] - P[:, 1], P[:, 0] - P[:, 2]], 1)
    l_max = np.linalg.norm(edges, axis=2).max(1)
    area = 0.5 * np.linalg.norm(np.cross(edges[:, 0], -edges[:, 2]), axis=1)
    return dist, l_max, l_max ** 2 / (2.0 * area)


def t_bar(t, dist, shape, cos):
    return (T_REL * t + T_COND * dist * shape) / np.maximum(np.abs(cos), 1e-3)


def uv_bar(spread, dist, shape, l_max, cos):
    return spread * (UV_REL + UV_COND * dist * shape / l_max) / np.maximum(np.abs(cos), 1e-3) \
        + UV_ABS
