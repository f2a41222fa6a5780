"""Pins the error bars of the ray-mesh hit (tests/meshbars.py) on the CPU.

The GPU kernels solve Moller-Trumbore in fp32.  Here the same solve is
emulated in numpy float32 (each operation rounded to fp32 as the kernels
round it, though without their fused multiply-adds, and with a correctly
rounded reciprocal where the kernels use the hardware's one-ulp one): the
fp32 pixel ray from the camera constants, the fp32 edges v1 - v0 and
v2 - v0, the determinant, the barycentrics and t, and the barycentric
interpolation of the vertex uv.  Over every pixel of the 24 seeded random
triangle soups that the oracle does not flag ambiguous, the emulated errors
against the oracle's fp64 hit must stay inside the bars, and the bars must
not be looser than 10x the largest emulated error (a bar that admits any
error says nothing)."""
import numpy as np
import pytest

import meshbars
import oracle
from randcfg import MESH_SEEDS, random_soup

f32 = np.float32


def _rays32(cams, W, H, pix):
    """The kernels' fp32 pixel rays: (origins, unit directions) [n, 3]."""
    view, rem = np.divmod(pix, H * W)
    j, i = np.divmod(rem, W)
    c = np.asarray(cams, np.float32).reshape(-1, 16)[view]
    half = 0.5 * c[:, 12].astype(np.float64) * np.pi / 180.0
    inv_f = (np.tan(half) / (0.5 * H)).astype(f32)
    cx = (i.astype(f32) + f32(0.5) - f32(0.5) * f32(W)) * inv_f
    cy = -((j.astype(f32) + f32(0.5) - f32(0.5) * f32(H)) * inv_f)
    d = np.stack([c[:, 0] * cx + c[:, 1] * cy - c[:, 2],
                  c[:, 4] * cx + c[:, 5] * cy - c[:, 6],
                  c[:, 8] * cx + c[:, 9] * cy - c[:, 10]], 1).astype(f32)
    inv = f32(1) / np.sqrt((d * d).sum(1, dtype=f32))
    return c[:, [3, 7, 11]], d * inv[:, None], view


def _cross(a, b):
    return np.stack([a[:, 1] * b[:, 2] - a[:, 2] * b[:, 1], a[:, 2] * b[:, 0] - a[:, 0] * b[:, 2],
                     a[:, 0] * b[:, 1] - a[:, 1] * b[:, 0]], 1)


def _dot(a, b):
    return a[:, 0] * b[:, 0] + a[:, 1] * b[:, 1] + a[:, 2] * b[:, 2]


def _solve32(o, d, v0, v1, v2):
    e1, e2 = v1 - v0, v2 - v0
    p = _cross(d, e2)
    inv = f32(1) / _dot(e1, p)
    s = o - v0
    b1 = _dot(s, p) * inv
    q = _cross(s, e1)
    b2 = _dot(d, q) * inv
    t = _dot(e2, q) * inv
    return t, b1, b2


@pytest.fixture(scope="module")
def emulated():
    rows = {"t_share": [], "uv_share": []}
    for seed in MESH_SEEDS:
        mesh, cams, W, H, _, _ = random_soup(seed)
        pix = np.arange(cams.shape[0] * H * W)
        g0, n, tri, amb = oracle.raycast_pixels(cams, W, H, mesh, pix,
                                                threads=oracle.max_threads())
        ok = (~amb) & (tri >= 0)
        if not ok.any():
            continue
        pix, tri, g0, n = pix[ok], tri[ok], g0[ok], n[ok]
        o, d, view = _rays32(cams, W, H, pix)
        P = np.asarray(mesh.positions, np.float32)[np.asarray(mesh.faces)[tri]]
        t, b1, b2 = _solve32(o, d, P[:, 0], P[:, 1], P[:, 2])
        d64 = np.array([oracle.camera_ray(cams[v], W, H, int(p % W), int((p // W) % H))[1]
                        for v, p in zip(view, pix)])
        cos = _dot(d64, n)
        origin = np.asarray(cams, np.float64).reshape(-1, 16)[view][:, [3, 7, 11]]
        dist, l_max, shape = meshbars.conditioning(mesh.positions, mesh.faces, tri, origin)
        dt = np.abs(t.astype(np.float64) - g0[:, 0])
        rows["t_share"].append(dt / meshbars.t_bar(g0[:, 0], dist, shape, cos))
        if mesh.uv is not None:
            UV = np.asarray(mesh.uv, np.float32)[np.asarray(mesh.faces)[tri]]
            b0 = f32(1) - b1 - b2
            uv = b0[:, None] * UV[:, 0] + b1[:, None] * UV[:, 1] + b2[:, None] * UV[:, 2]
            du = np.abs(uv.astype(np.float64) - g0[:, 1:3]).max(1)
            spread = (UV.max(1) - UV.min(1)).max(1).astype(np.float64)
            rows["uv_share"].append(du / meshbars.uv_bar(spread, dist, shape, l_max, cos))
    return {k: np.concatenate(v) for k, v in rows.items()}


def test_t_bar_holds_and_is_tight(emulated):
    share = emulated["t_share"]
    print(f"t: {share.size} px, largest share of the bar {share.max():.3f}")
    assert share.size > 10000
    assert share.max() <= 1.0, share.max()
    assert share.max() >= 0.1, share.max()


def test_uv_bar_holds_and_is_tight(emulated):
    share = emulated["uv_share"]
    print(f"uv: {share.size} px, largest share of the bar {share.max():.3f}")
    assert share.size > 5000
    assert share.max() <= 1.0, share.max()
    assert share.max() >= 0.1, share.max()
