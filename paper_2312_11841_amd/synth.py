"""Seeded synthetic inputs shaped like the MixRT workloads.

This module only *draws* inputs: G-buffers, cameras, displacement textures,
hash tables and MLP weights.  It holds none of the rendering arithmetic (no
pixel-to-ray mapping, displacement, contraction, hashing, MLP or compositing),
so both the HIP path and the CPU oracle can consume its arrays without sharing
any of the method's code.

The paper measures on trained indoor Unbounded-360 scenes rendered at
1280x720 (Sec. 5.1.1); neither the dataset nor trained assets are available, so
these generators stand in for them with the same shapes: an indoor room seen
from inside (depths 0.5-20), a texture atlas addressed by per-surface UV
charts, hash tables and MLPs with the sizes listed per configuration.

Screen-space room: every visible surface of the procedural room is planar, and
a planar surface seen through any pinhole camera has an inverse depth that is
affine in the pixel coordinates.  The generator therefore writes inverse depth
directly as an affine function of normalised screen coordinates and keeps the
nearest surface per pixel.  This gives the spatial coherence of a rasterised
G-buffer (adjacent pixels hit adjacent points) without evaluating any camera
ray.
"""
from __future__ import annotations

import dataclasses
import hashlib
from dataclasses import dataclass, field

import numpy as np

# Data-type codes shared with the C ABI descriptor fields (values, not code).
DT_F32 = 0
DT_F16 = 1
DT_U8 = 2

_DT_CODE = {"f32": DT_F32, "f16": DT_F16, "u8": DT_U8}
_NP_DT = {"f32": np.float32, "f16": np.float16, "u8": np.uint8}


@dataclass(frozen=True)
class SceneConfig:
    """One workload: image size, sampling, texture, hash grid and MLP shapes."""

    name: str
    views: int
    H: int
    W: int
    K: int
    delta: float
    gbuf: str                 # "iid" (cache-hostile), "room" (coherent) or
                              # "mesh" (computed from `mesh_seed`'s mesh)
    tex_R: int
    tex_V: int
    tex_dtype: str            # "f32" | "f16"
    tex_range: float          # texture values ~ U[-tex_range, tex_range]
    L: int
    log2_T: int
    F: int
    N_min: int
    N_max: int
    table_dtype: str          # "f32" | "f16"
    table_range: float        # table values ~ U[-table_range, table_range]
    widths: tuple             # (in, hidden..., 4); (in,) = the MLP removed
    view_sh_dim: int          # 0 or 16
    w_std: float              # weights ~ N(0, w_std), stored fp16
    seed: int
    fov_y_deg: float = 60.0
    t_term: float = 1e-4
    head_scale: float = 1.0   # multiplies the output-layer weights
    sigma_gain: float = 0.0   # > 0: the head's density weights become
                              # sigma_gain * |w| (opaque content)
    bg: tuple = (0.0, 0.0, 0.0)
    rows: int = 0             # >0: keep only the first `rows` image rows
    disp: str = "ray"         # "ray": scalar along the ray; "vec3": Eq. 2 as
                              # printed (SH vector x scale map); "none"
    sh_degree: int = 0        # "vec3": SH degree D, 3 (D+1)^2 channels
    scale_range: tuple = (0.0, 1.0)  # "vec3": scale map values
    mesh_seed: int = -1       # "mesh": seed of make_mesh
    mesh_args: tuple = ()     # "mesh": other make_mesh arguments, (name, value) pairs

    @property
    def T(self) -> int:
        return 1 << self.log2_T

    @property
    def rays(self) -> int:
        return self.views * self.rows_kept * self.W

    @property
    def rows_kept(self) -> int:
        return self.rows if self.rows else self.H

    @property
    def samples(self) -> int:
        return self.rays * self.K

    @property
    def tex_channels(self) -> int:
        """Channels the displacement form reads."""
        if self.disp == "vec3":
            return 3 * (self.sh_degree + 1) ** 2
        return self.tex_V if self.disp == "ray" else 0

    @property
    def tex_C(self) -> int:
        """Stored channels per texel: the used ones padded to 16-byte texels."""
        eb = {"f32": 4, "f16": 2, "u8": 1}[self.tex_dtype]
        per = 16 // eb
        n = max(self.tex_channels, 1)
        return n if self.disp == "ray" else -(-n // per) * per

    def replace(self, **kw) -> "SceneConfig":
        return dataclasses.replace(self, **kw)


# --- the workloads -----------------------------------------------------------

TINY64 = SceneConfig(
    name="tiny64", views=1, H=64, W=64, K=4, delta=0.01, gbuf="iid",
    tex_R=64, tex_V=4, tex_dtype="f32", tex_range=0.05,
    L=8, log2_T=14, F=2, N_min=16, N_max=256, table_dtype="f32",
    table_range=1e-2, widths=(16, 32, 4), view_sh_dim=0, w_std=0.1, seed=1)

# Same shapes, but densities and features large enough that every sample
# matters: alpha in roughly [0.1, 0.99] per sample, colours spread over (0,1).
TINY64_DENSE = TINY64.replace(name="tiny64_dense", delta=0.5, table_range=1.0,
                              head_scale=8.0, bg=(0.2, 0.4, 0.6), seed=11)

VIEW720P = SceneConfig(
    name="view720p", views=1, H=720, W=1280, K=8, delta=0.01, gbuf="room",
    tex_R=1024, tex_V=8, tex_dtype="f16", tex_range=0.05,
    L=16, log2_T=19, F=2, N_min=16, N_max=4096, table_dtype="f16",
    table_range=1e-2, widths=(48, 64, 64, 4), view_sh_dim=16, w_std=0.05,
    seed=2)

VIEW720P_DENSE = VIEW720P.replace(name="view720p_dense", delta=0.25,
                                  table_range=1.0, w_std=0.2, head_scale=2.0,
                                  bg=(0.2, 0.4, 0.6), seed=12)

# Opaque content: view720p with the density head's weights made positive
# and large, so a ray's first samples are nearly opaque and it reaches the
# early-termination transmittance within a few samples, as at a solid
# surface (about 2.6 of its 8 samples on average, counted with the oracle's
# densities); the colours stay view720p's.  The translucent variant stops
# later and more spread out (about 6 of 8 samples, a quarter of the rays
# never stop).
OPAQUE720P = VIEW720P.replace(name="opaque720p", sigma_gain=400.0, bg=(0.2, 0.4, 0.6), seed=21)
TRANSLUCENT720P = OPAQUE720P.replace(name="translucent720p", sigma_gain=300.0)

BATCH8X1080P = VIEW720P.replace(name="batch8x1080p", views=8, H=1080, W=1920,
                                log2_T=21, N_max=8192, seed=3)


def sweep_config(rays: int, K: int, dense: bool = False) -> SceneConfig:
    """First `rays` rays of a coherent 4096x4096 view, on the 720p grid/MLP."""
    assert rays % 4096 == 0
    base = VIEW720P_DENSE if dense else VIEW720P
    return base.replace(name=f"sweep_r{rays}_k{K}" + ("_dense" if dense else ""),
                        H=4096, W=4096, rows=rays // 4096, K=K, seed=4)


# The deployed grid of the paper's implementation details: four levels,
# resolution 256 to 4096, 2^21 entries of four features, one query per pixel.
# With one query per pixel the density saturates (delta = 10), so the pixel
# is the MLP's colour, as in the paper's pipeline.
DEPLOYED720P = VIEW720P.replace(name="deployed720p", K=1, delta=10.0, L=4, log2_T=21, F=4,
                                N_min=256, N_max=4096, widths=(32, 64, 64, 4),
                                seed=5)

# The paper's deployed configuration with Eq. 2 as printed: SH degree 2
# displacement vectors (27 channels, stored in 32-byte texels) times a scale
# map, both 8-bit at R_m = 1536 (Sec. 4.3.2, Sec. 5.1.2), the deployed grid,
# one query per pixel.  Features and weights large enough for a structured
# frame (rgb over ~[0.3, 0.6]) while the fp16 MLP inputs stay well inside the
# frame tolerance.
PAPER720P = DEPLOYED720P.replace(name="paper720p", tex_R=1536, tex_dtype="u8", disp="vec3",
                                 sh_degree=2, tex_range=0.05, scale_range=(0.0, 1.0),
                                 table_range=0.5, w_std=0.2, head_scale=1.0,
                                 bg=(0.2, 0.4, 0.6), seed=6)

# Tiny workloads for the other displacement forms (CPU-checkable).
TINY64_VEC3 = TINY64_DENSE.replace(name="tiny64_vec3", disp="vec3", sh_degree=1,
                                   tex_range=0.2, seed=13)
TINY64_U8 = TINY64_DENSE.replace(name="tiny64_u8", tex_dtype="u8", tex_range=0.3, seed=14)
TINY64_NODISP = TINY64_DENSE.replace(name="tiny64_nodisp", disp="none", seed=15)

# Tab. 6's ablation: the paper's configuration without the displacement map.
PAPER720P_NOVDD = PAPER720P.replace(name="paper720p_novdd", disp="none")


def table3_config(L: int, log2_T: int, mlp: bool) -> SceneConfig:
    """Tab. 3's profiling points: one query per pixel, no displacement map, F=4
    entries over the deployed 256..4096 resolutions, with the MLP (two hidden
    layers of 8 neurons, as the table gives it) or without it (level
    features summed per component)."""
    widths = (L * 4, 8, 8, 4) if mlp else (L * 4,)
    return PAPER720P.replace(name=f"tab3_L{L}_T{log2_T}" + ("_mlp" if mlp else ""), disp="none",
                             L=L, log2_T=log2_T, view_sh_dim=0, widths=widths, seed=7)


TABLE3 = [table3_config(8, 17, True), table3_config(8, 17, False), table3_config(1, 17, False),
          table3_config(8, 5, False), table3_config(8, 22, False)]
LEVEL_SWEEP = [table3_config(L, 17, False) for L in (1, 2, 4, 8, 16)]
# Table size at L = 8: Tab. 3's 2^5, 2^17 and 2^22, and the deployed 2^21.
SIZE_SWEEP = [table3_config(8, t, False) for t in (5, 17, 21, 22)]

# The whole pipeline including geometry: a seeded 499,712-triangle mesh (a
# perturbed-sphere room of radius 6 with 24 perturbed spheres and 16 boxes,
# 11 MB) turned into the G-buffer per frame, then view720p's displacement,
# grid, MLP and compositing at 1280x720.
MESH720P = VIEW720P.replace(name="mesh720p", gbuf="mesh", mesh_seed=7)
# Small enough for the oracle's brute-force ray casting of every pixel
# (1,280 + 6 x 320 + 4 x 108 = 3,632 triangles).
TINY64_MESH = TINY64_DENSE.replace(
    name="tiny64_mesh", gbuf="mesh", mesh_seed=8, seed=16,
    mesh_args=(("room_level", 3), ("n_objects", 6), ("object_level", 2), ("n_boxes", 4),
               ("box_div", 3)))

CONFIGS = {c.name: c for c in (TINY64, TINY64_DENSE, VIEW720P, VIEW720P_DENSE, OPAQUE720P,
                               TRANSLUCENT720P,
                               BATCH8X1080P, DEPLOYED720P, PAPER720P, PAPER720P_NOVDD,
                               TINY64_VEC3, TINY64_U8, TINY64_NODISP, MESH720P, TINY64_MESH,
                               *TABLE3, *LEVEL_SWEEP, *SIZE_SWEEP)}


# --- scene container ----------------------------------------------------------

@dataclass
class Scene:
    cfg: SceneConfig
    g0: np.ndarray            # [views, rows, W, 4] f32: (t, u, v, 0)
    g1: np.ndarray            # [views, rows, W, 4] f32: (nx, ny, nz, 0)
    cams: np.ndarray          # [views, 16] f32: c2w row-major 3x4, fov_y_deg, bg rgb
    tex: np.ndarray           # [R, R, C] f32/f16/u8 (C stored channels)
    table: np.ndarray         # [L, T, F] f32/f16
    weights: list             # per layer [in, out] f16
    scale: np.ndarray = None  # [R, R] scale map ("vec3"), same dtype as tex
    q_scale: tuple = (0.0, 0.0)   # 8-bit maps: value = q_offset + q_scale * q
    q_offset: tuple = (0.0, 0.0)  # ([0] coefficient map, [1] scale map)
    extra: dict = field(default_factory=dict)
    mesh: "Mesh" = None       # "mesh" workloads: the geometry; g0/g1 then hold
                              # misses until a ray cast fills them

    @property
    def weights_flat(self) -> np.ndarray:
        if not self.weights:
            return np.zeros(0, np.float16)
        return np.concatenate([w.reshape(-1) for w in self.weights]).astype(np.float16)

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.g0, self.g1, self.cams, self.tex, self.table, self.weights_flat,
                  self.scale if self.scale is not None else np.zeros(0)):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()


def _rot_y(deg: float) -> np.ndarray:
    a = np.deg2rad(deg)
    c, s = np.cos(a), np.sin(a)
    return np.array([[c, 0, s], [0, 1, 0], [-s, 0, c]])


def _rot_x(deg: float) -> np.ndarray:
    a = np.deg2rad(deg)
    c, s = np.cos(a), np.sin(a)
    return np.array([[1, 0, 0], [0, c, -s], [0, s, c]])


def _camera_rows(cfg: SceneConfig, rng: np.random.Generator) -> np.ndarray:
    cams = np.zeros((cfg.views, 16), np.float32)
    for v in range(cfg.views):
        if cfg.gbuf == "iid":
            R = np.eye(3)
            o = np.zeros(3)
        elif cfg.views == 1:
            R = _rot_y(15.0) @ _rot_x(-5.0)
            o = np.array([0.3, 0.2, -0.1])
        else:  # a 360-degree capture pattern: poses on a circle, facing out
            yaw = 360.0 * v / cfg.views
            R = _rot_y(yaw) @ _rot_x(-5.0)
            o = 0.5 * np.array([np.sin(np.deg2rad(yaw)), 0.0, np.cos(np.deg2rad(yaw))])
            o[1] = 0.2
        c2w = np.concatenate([R, o[:, None]], axis=1)
        cams[v, :12] = c2w.reshape(-1)
        cams[v, 12] = cfg.fov_y_deg
        cams[v, 13:16] = cfg.bg
    return cams


def _iid_gbuffer(cfg: SceneConfig, rng: np.random.Generator):
    n = cfg.views * cfg.rows_kept * cfg.W
    g0 = np.zeros((n, 4), np.float32)
    g0[:, 0] = rng.uniform(1.0, 4.0, n)
    g0[:, 1:3] = rng.uniform(0.0, 1.0, (n, 2))
    g1 = np.zeros((n, 4), np.float32)
    g1[:, 2] = 1.0  # facing a camera that looks down -z
    shape = (cfg.views, cfg.rows_kept, cfg.W, 4)
    return g0.reshape(shape), g1.reshape(shape)


def _room_view(rng: np.random.Generator, H: int, W: int, rows: int):
    """One screen-space indoor view: walls, floor, ceiling, boxes, blobs."""
    jj, ii = np.mgrid[0:rows, 0:W].astype(np.float64)
    xs = (ii + 0.5 - W / 2) / (H / 2)          # horizontal, aspect-scaled
    ys = (jj + 0.5 - H / 2) / (H / 2)          # vertical, +1 at the bottom
    # Room surfaces: inverse depth affine in (xs, ys); the nearest wins.
    back = 1.0 / rng.uniform(8.0, 18.0)
    kf, kc = rng.uniform(0.5, 0.9), rng.uniform(0.3, 0.6)
    kl, kr = rng.uniform(0.25, 0.5), rng.uniform(0.25, 0.5)
    yh = rng.uniform(-0.15, 0.15)
    xh = rng.uniform(-0.2, 0.2)
    surf_inv = np.stack([
        np.full_like(xs, back),                # back wall
        kf * (ys - yh),                        # floor
        -kc * (ys - yh),                       # ceiling
        -kl * (xs - xh),                       # left wall
        kr * (xs - xh),                        # right wall
    ])
    normals = np.array([[0, 0, 1], [0, 1, 0], [0, -1, 0], [1, 0, 0], [-1, 0, 0]],
                       np.float64)
    sid = np.argmax(surf_inv, axis=0)
    inv = np.take_along_axis(surf_inv, sid[None], 0)[0]
    nrm = normals[sid]
    # Per-surface UV charts: affine in screen space, wrapped into [0, 1).
    coef = rng.uniform(-0.6, 0.6, (5, 2, 3))
    u = np.zeros_like(xs)
    v = np.zeros_like(xs)
    for s in range(5):
        m = sid == s
        u[m] = coef[s, 0, 0] * xs[m] + coef[s, 0, 1] * ys[m] + coef[s, 0, 2]
        v[m] = coef[s, 1, 0] * xs[m] + coef[s, 1, 1] * ys[m] + coef[s, 1, 2]
    aspect = W / H
    # Boxes: planar screen rectangles nearer than the room.
    for _ in range(int(rng.integers(6, 12))):
        cx, cy = rng.uniform(-aspect, aspect), rng.uniform(-0.6, 0.9)
        hw, hh = rng.uniform(0.05, 0.4), rng.uniform(0.05, 0.4)
        a0 = 1.0 / rng.uniform(0.6, 6.0)
        ax, ay = rng.uniform(-0.1, 0.1, 2) * a0
        binv = a0 + ax * (xs - cx) + ay * (ys - cy)
        m = (np.abs(xs - cx) < hw) & (np.abs(ys - cy) < hh) & (binv > inv)
        inv[m] = binv[m]
        c = rng.uniform(-1.0, 1.0, (2, 3))
        u[m] = c[0, 0] * xs[m] + c[0, 1] * ys[m] + c[0, 2]
        v[m] = c[1, 0] * xs[m] + c[1, 1] * ys[m] + c[1, 2]
        n = rng.normal(size=3)
        n[2] = abs(n[2]) + 1.0
        nrm[m] = n / np.linalg.norm(n)
    # Perturbed blobs: screen disks with a bulging inverse depth.
    for _ in range(int(rng.integers(2, 5))):
        cx, cy = rng.uniform(-aspect, aspect), rng.uniform(-0.5, 0.8)
        rad = rng.uniform(0.08, 0.35)
        t0 = rng.uniform(0.8, 5.0)
        rho2 = ((xs - cx) ** 2 + (ys - cy) ** 2) / rad ** 2
        wob = 1.0 + 0.05 * np.sin(7.0 * np.arctan2(ys - cy, xs - cx))
        inside = rho2 < wob ** 2
        bulge = np.sqrt(np.clip(1.0 - rho2 / wob ** 2, 0.0, 1.0))
        binv = 1.0 / (t0 - 0.4 * t0 * rad * bulge)
        m = inside & (binv > inv)
        inv[m] = binv[m]
        u[m] = 0.5 + 0.5 * (xs[m] - cx) / rad
        v[m] = 0.5 + 0.5 * (ys[m] - cy) / rad
        nz = np.maximum(bulge[m], 1e-3)
        nn = np.stack([(xs[m] - cx) / rad, -(ys[m] - cy) / rad, nz], -1)
        nrm[m] = nn / np.linalg.norm(nn, axis=-1, keepdims=True)
    with np.errstate(divide="ignore"):
        t = np.clip(1.0 / np.maximum(inv, 1e-9), 0.5, 20.0)
    u = u - np.floor(u)
    v = v - np.floor(v)
    g0 = np.stack([t, u, v, np.zeros_like(t)], -1).astype(np.float32)
    g1 = np.concatenate([nrm, np.zeros_like(t)[..., None]], -1).astype(np.float32)
    return g0, g1


def _room_gbuffer(cfg: SceneConfig, rng: np.random.Generator):
    g0s, g1s = [], []
    for _ in range(cfg.views):
        a, b = _room_view(rng, cfg.H, cfg.W, cfg.rows_kept)
        g0s.append(a)
        g1s.append(b)
    return np.stack(g0s), np.stack(g1s)


def make_scene(cfg: SceneConfig) -> Scene:
    """Draw every input of `cfg` in a fixed order: G-buffer, camera, texture,
    table, weights."""
    rng = np.random.default_rng(cfg.seed)
    mesh = None
    if cfg.gbuf == "iid":
        g0, g1 = _iid_gbuffer(cfg, rng)
    elif cfg.gbuf == "mesh":
        mesh = make_mesh(cfg.mesh_seed, **dict(cfg.mesh_args))
        shape = (cfg.views, cfg.rows_kept, cfg.W, 4)
        g0 = np.zeros(shape, np.float32)
        g0[..., 0] = -1.0
        g1 = np.zeros(shape, np.float32)
    else:
        g0, g1 = _room_gbuffer(cfg, rng)
    cams = _camera_rows(cfg, rng)
    shape = (cfg.tex_R, cfg.tex_R, cfg.tex_C)
    q_scale, q_offset = (0.0, 0.0), (0.0, 0.0)
    scale = None
    if cfg.tex_dtype == "u8":
        lo, hi = cfg.scale_range
        q_scale = (2.0 * cfg.tex_range / 255.0, (hi - lo) / 255.0)
        q_offset = (-cfg.tex_range, lo)
        tex = rng.integers(0, 256, shape, dtype=np.uint8)
        if cfg.disp == "vec3":
            scale = rng.integers(0, 256, shape[:2], dtype=np.uint8)
    else:
        tex = rng.uniform(-cfg.tex_range, cfg.tex_range, shape).astype(_NP_DT[cfg.tex_dtype])
        if cfg.disp == "vec3":
            scale = rng.uniform(*cfg.scale_range, shape[:2]).astype(_NP_DT[cfg.tex_dtype])
    table = rng.uniform(-cfg.table_range, cfg.table_range,
                        (cfg.L, cfg.T, cfg.F)).astype(np.float32)
    table = table.astype(_NP_DT[cfg.table_dtype])
    assert cfg.widths[0] == cfg.L * cfg.F + cfg.view_sh_dim
    assert cfg.widths[-1] == 4 or len(cfg.widths) == 1
    weights = []
    for m in range(len(cfg.widths) - 1):
        w = rng.normal(0.0, cfg.w_std, (cfg.widths[m], cfg.widths[m + 1]))
        if m == len(cfg.widths) - 2:
            w = w * cfg.head_scale
            if cfg.sigma_gain > 0:
                w[:, 0] = cfg.sigma_gain * np.abs(w[:, 0])
        weights.append(w.astype(np.float16))
    return Scene(cfg=cfg, g0=np.ascontiguousarray(g0), g1=np.ascontiguousarray(g1),
                 cams=cams, tex=np.ascontiguousarray(tex),
                 table=np.ascontiguousarray(table), weights=weights,
                 scale=None if scale is None else np.ascontiguousarray(scale),
                 q_scale=q_scale, q_offset=q_offset, mesh=mesh)


def dtype_code(name: str) -> int:
    return _DT_CODE[name]


# --- procedural low-poly mesh (the G-buffer's geometry) -----------------------

def _icosphere(level: int):
    """Unit icosphere: 20 * 4^level faces (vertices deduplicated per level)."""
    t = (1.0 + 5 ** 0.5) / 2.0
    v = np.array([[-1, t, 0], [1, t, 0], [-1, -t, 0], [1, -t, 0], [0, -1, t], [0, 1, t],
                  [0, -1, -t], [0, 1, -t], [t, 0, -1], [t, 0, 1], [-t, 0, -1], [-t, 0, 1]],
                 np.float64)
    f = np.array([[0, 11, 5], [0, 5, 1], [0, 1, 7], [0, 7, 10], [0, 10, 11], [1, 5, 9],
                  [5, 11, 4], [11, 10, 2], [10, 7, 6], [7, 1, 8], [3, 9, 4], [3, 4, 2],
                  [3, 2, 6], [3, 6, 8], [3, 8, 9], [4, 9, 5], [2, 4, 11], [6, 2, 10],
                  [8, 6, 7], [9, 8, 1]], np.int64)
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    for _ in range(level):
        edges = np.concatenate([f[:, [0, 1]], f[:, [1, 2]], f[:, [2, 0]]])
        key = np.sort(edges, axis=1)
        uniq, inv = np.unique(key, axis=0, return_inverse=True)
        mid = v[uniq[:, 0]] + v[uniq[:, 1]]
        mid /= np.linalg.norm(mid, axis=1, keepdims=True)
        m = inv.reshape(3, -1).T + len(v)           # midpoints of edges 01, 12, 20
        v = np.concatenate([v, mid])
        a, b, c = f[:, 0], f[:, 1], f[:, 2]
        m01, m12, m20 = m[:, 0], m[:, 1], m[:, 2]
        f = np.concatenate([np.stack([a, m01, m20], 1), np.stack([b, m12, m01], 1),
                            np.stack([c, m20, m12], 1), np.stack([m01, m12, m20], 1)])
    return v, f


@dataclass
class Mesh:
    positions: np.ndarray   # [nv, 3] f32
    faces: np.ndarray       # [nf, 3] i32
    uv: np.ndarray          # [nv, 2] f32, texture atlas coordinates in [0, 1]

    @property
    def nbytes(self) -> int:
        return self.positions.nbytes + self.faces.nbytes + self.uv.nbytes


def _box(div: int):
    """Cube [-1, 1]^3, each face a div x div grid of quads split in two,
    wound so that e1 x e2 points out; returns positions, faces and each
    vertex's (face index, s, t) chart coordinates in [0, 1]^2."""
    g = np.linspace(-1.0, 1.0, div + 1)
    S, T = np.meshgrid(g, g, indexing="ij")
    pos, faces, chart = [], [], []
    for k, (ax, sign) in enumerate([(a, s) for a in range(3) for s in (1.0, -1.0)]):
        p = np.zeros((div + 1, div + 1, 3))
        p[..., ax] = sign
        p[..., (ax + 1) % 3] = S
        p[..., (ax + 2) % 3] = T
        idx = np.arange((div + 1) ** 2).reshape(div + 1, div + 1) + k * (div + 1) ** 2
        q00, q10 = idx[:-1, :-1].ravel(), idx[1:, :-1].ravel()
        q11, q01 = idx[1:, 1:].ravel(), idx[:-1, 1:].ravel()
        f = np.concatenate([np.stack([q00, q10, q11], 1), np.stack([q00, q11, q01], 1)])
        faces.append(f if sign > 0 else f[:, ::-1])
        pos.append(p.reshape(-1, 3))
        chart.append(np.stack([np.full(S.size, k), (S.ravel() + 1) / 2, (T.ravel() + 1) / 2], 1))
    return np.concatenate(pos), np.concatenate(faces), np.concatenate(chart)


def _rotation(rng: np.random.Generator) -> np.ndarray:
    q = rng.normal(size=4)
    w, x, y, z = q / np.linalg.norm(q)
    return np.array([[1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
                     [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
                     [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)]])


def make_mesh(seed: int, room_level: int = 7, n_objects: int = 24, object_level: int = 4,
              n_boxes: int = 16, box_div: int = 16, room_radius: float = 6.0) -> Mesh:
    """A perturbed-sphere room seen from inside, with perturbed-sphere and box
    objects placed clear of a 0.8-radius ball around the origin (where the
    cameras stand).  Defaults: 499,712 triangles.

    Texture atlas: the room takes the [0, 0.5]^2 quarter with a spherical
    (azimuth, polar) chart; every object takes one 0.125-sized tile (spheres:
    spherical chart, boxes: a 3 x 2 grid of face charts)."""
    rng = np.random.default_rng(seed)
    tiles = [(0.5 + (k % 4) * 0.125, (k // 4) * 0.125) for k in range(32)] + \
            [((k % 4) * 0.125, 0.5 + (k // 4) * 0.125) for k in range(32)]
    pos, faces, uvs = [], [], []
    base = 0

    def place(reach):
        while True:
            c = rng.uniform(-0.6, 0.6, 3) * room_radius
            if reach + 0.8 < np.linalg.norm(c) < 0.75 * room_radius:
                return c

    for o in range(1 + n_objects + n_boxes):
        if o <= n_objects:
            v, f = _icosphere(room_level if o == 0 else object_level)
            amp = 0.06 if o == 0 else 0.12
            r0 = room_radius if o == 0 else rng.uniform(0.2, 0.8)
            c = np.zeros(3) if o == 0 else place(r0 * (1 + amp))
            th = np.arccos(np.clip(v[:, 2], -1, 1))
            ph = np.arctan2(v[:, 1], v[:, 0])
            k1, k2 = rng.integers(2, 6, 2)
            ph0 = rng.uniform(0, 2 * np.pi)
            r = r0 * (1.0 + amp * np.sin(k1 * th) * np.cos(k2 * ph + ph0))
            p = c + v * r[:, None]
            cu, cv = (ph + np.pi) / (2 * np.pi), th / np.pi
            if o == 0:
                uv = np.stack([0.5 * cu, 0.5 * cv], 1)
            else:
                tu, tv = tiles[(o - 1) % len(tiles)]
                uv = np.stack([tu + 0.125 * cu, tv + 0.125 * cv], 1)
        else:
            v, f, chart = _box(box_div)
            half = rng.uniform(0.15, 0.6, 3)
            R = _rotation(rng)
            c = place(float(np.linalg.norm(half)))
            p = c + (v * half) @ R.T
            tu, tv = tiles[(o - 1) % len(tiles)]
            k = chart[:, 0]
            cell = 0.125 / 3
            uv = np.stack([tu + (k % 3 + chart[:, 1]) * cell, tv + (k // 3 + chart[:, 2]) * cell], 1)
        pos.append(p)
        uvs.append(uv)
        faces.append(f + base)
        base += len(p)
    return Mesh(positions=np.concatenate(pos).astype(np.float32),
                faces=np.concatenate(faces).astype(np.int32),
                uv=np.clip(np.concatenate(uvs), 0, 1).astype(np.float32))
