"""Seeded random workloads for the parity sweep: every combination the library
builds a render kernel for (displacement form and storage, F, table dtype, MLP
shape), with the remaining parameters drawn at random inside the supported
ranges (samples per ray, spacing, table size, level resolutions, views, ragged
image sizes, G-buffer kind, cameras, misses, background, termination)."""
import numpy as np

from paper_2312_11841_amd import synth

TEX = {
    "f32_ray": dict(tex_dtype="f32", disp="ray"),
    "f16_ray": dict(tex_dtype="f16", disp="ray"),
    "u8_ray": dict(tex_dtype="u8", disp="ray"),
    "f16_vec3_d2": dict(tex_dtype="f16", disp="vec3", sh_degree=2),
    "u8_vec3_d2": dict(tex_dtype="u8", disp="vec3", sh_degree=2),
    "f32_vec3_d1": dict(tex_dtype="f32", disp="vec3", sh_degree=1),
    "none": dict(tex_dtype="f32", disp="none"),
    # Eq. 2 as printed at a random SH degree 0..3 (the kernels that take the
    # degree at run time)
    "f32_vec3": dict(tex_dtype="f32", disp="vec3"),
    "f16_vec3": dict(tex_dtype="f16", disp="vec3"),
    "u8_vec3": dict(tex_dtype="u8", disp="vec3"),
}

# (displacement, F, fp16 table, MLP in, hidden, hidden layers); 0, 0, 0 = the
# MLP removed, any input width
BUILT = [
    ("f32_ray", 2, False, 16, 32, 1), ("f32_ray", 2, False, 32, 32, 1),
    ("f16_ray", 2, True, 48, 64, 2), ("f16_ray", 2, True, 32, 64, 2),
    ("f16_ray", 4, True, 32, 64, 2), ("f16_ray", 4, True, 16, 64, 2),
    ("u8_vec3_d2", 4, True, 32, 64, 2), ("f16_vec3_d2", 4, True, 32, 64, 2),
    ("f32_vec3_d1", 2, False, 16, 32, 1), ("u8_ray", 2, False, 16, 32, 1),
    ("none", 2, False, 16, 32, 1), ("none", 2, True, 48, 64, 2),
    ("none", 4, True, 32, 64, 2), ("none", 4, True, 32, 16, 2),
    ("none", 4, True, 0, 0, 0), ("none", 2, False, 0, 0, 0),
    ("f32_ray", 2, False, 0, 0, 0), ("u8_vec3_d2", 4, True, 0, 0, 0),
    ("f32_vec3", 2, False, 16, 32, 1), ("f16_vec3", 2, False, 16, 32, 1),
    ("u8_vec3", 2, False, 16, 32, 1), ("f32_vec3", 4, True, 32, 64, 2),
    ("f16_vec3", 4, True, 32, 64, 2), ("u8_vec3", 4, True, 32, 64, 2),
    ("none", 4, True, 32, 8, 2),   # hidden width 8 on the 16-wide tile
]

SEEDS = list(range(1000, 1050))


def _random_rotation(rng: np.random.Generator) -> np.ndarray:
    """A uniformly random rotation matrix (from a normalised Gaussian quaternion)."""
    w, x, y, z = (q := rng.normal(size=4)) / np.linalg.norm(q)
    return np.array([[1 - 2 * (y * y + z * z), 2 * (x * y - w * z), 2 * (x * z + w * y)],
                     [2 * (x * y + w * z), 1 - 2 * (x * x + z * z), 2 * (y * z - w * x)],
                     [2 * (x * z - w * y), 2 * (y * z + w * x), 1 - 2 * (x * x + y * y)]])


def random_config(seed: int) -> synth.SceneConfig:
    rng = np.random.default_rng(seed)
    tex, F, f16, m_in, hid, nhid = BUILT[seed % len(BUILT)]
    if nhid:
        views_sh = [v for v in (0, 16) if m_in - v >= F and (m_in - v) % F == 0
                    and (m_in - v) // F <= 32]
        view_sh = int(rng.choice(views_sh))
        L = (m_in - view_sh) // F
        widths = (m_in,) + (hid,) * nhid + (4,)
    else:
        view_sh = 0
        Ls = [L for L in range(1, 25) if (L * F) % 4 == 0]
        L = int(rng.choice(Ls))
        widths = (L * F,)
    n_min = int(rng.integers(2, 41))
    n_max = int(min(2048, n_min * rng.uniform(1.0, 64.0)))
    H, W = int(rng.integers(1, 38)), int(rng.integers(1, 42))
    tex_kw = dict(TEX[tex])
    if tex_kw["disp"] == "vec3" and "sh_degree" not in tex_kw:
        tex_kw["sh_degree"] = int(rng.integers(0, 4))
    return synth.TINY64.replace(
        name=f"rand{seed}", views=int(rng.integers(1, 4)), H=H, W=W,
        K=int(rng.choice([1, 2, 3, 4, 5, 7, 8, 13, 16, 32, 64])),
        delta=float(rng.uniform(0.002, 0.3)),
        gbuf=str(rng.choice(["iid", "room"])),
        tex_R=int(rng.integers(1, 49)), tex_V=int(rng.integers(1, 17)),
        tex_range=float(rng.uniform(0.02, 0.3)), **tex_kw,
        L=L, log2_T=int(rng.integers(6, 18)), F=F, N_min=n_min, N_max=n_max,
        table_dtype="f16" if f16 else "f32", table_range=float(rng.uniform(0.01, 0.5)),
        widths=widths, view_sh_dim=view_sh, w_std=float(rng.uniform(0.03, 0.12)),
        head_scale=float(rng.uniform(0.5, 3.0)),
        fov_y_deg=float(rng.uniform(20.0, 120.0)),
        t_term=float(rng.choice([0.0, 1e-4, 1e-2])),
        bg=tuple(float(b) for b in rng.uniform(0.0, 1.0, 3)), seed=seed)


def random_scene(cfg: synth.SceneConfig) -> synth.Scene:
    """The workload's scene with each camera posed at random and about 5% of
    the pixels turned into misses (t of -1, 0, NaN or +inf)."""
    sc = synth.make_scene(cfg)
    rng = np.random.default_rng(cfg.seed + 7919)
    for v in range(cfg.views):
        R = _random_rotation(rng)
        o = rng.uniform(-1.0, 1.0, 3)
        sc.cams[v, :12] = np.concatenate([R, o[:, None]], axis=1).reshape(-1).astype(np.float32)
    flat = sc.g0.reshape(-1, 4)
    miss = rng.random(flat.shape[0]) < 0.05
    flat[miss, 0] = rng.choice(np.array([-1.0, 0.0, np.nan, np.inf], np.float32), miss.sum())
    return sc


# --- random triangle soups for the geometry stage --------------------------

MESH_SEEDS = list(range(2000, 2024))


def random_soup(seed: int):
    """A seeded triangle soup mixing small, sliver, huge, near-camera and
    degenerate (a repeated vertex) triangles, with or without uv, and the
    cameras, image size and grid options to view it with."""
    rng = np.random.default_rng(seed)
    n = int(np.exp(rng.uniform(0.0, np.log(3000.0))))
    kinds = rng.choice(5, n, p=[0.55, 0.15, 0.1, 0.1, 0.1])
    tris = np.zeros((n, 3, 3))
    for t in range(n):
        c = rng.uniform(-4.0, 4.0, 3)
        if kinds[t] == 0:                               # small
            tris[t] = c + rng.normal(0.0, rng.uniform(0.01, 0.3), (3, 3))
        elif kinds[t] == 1:                             # sliver: one short edge
            a, b = c, c + rng.normal(0.0, 0.5, 3)
            tris[t] = [a, b, b + rng.normal(0.0, 1e-3, 3)]
        elif kinds[t] == 2:                             # huge
            tris[t] = c + rng.normal(0.0, rng.uniform(5.0, 40.0), (3, 3))
        elif kinds[t] == 3:                             # close to the cameras
            tris[t] = rng.normal(0.0, rng.uniform(0.02, 0.3), 3) + rng.normal(0.0, 0.1, (3, 3))
        else:                                           # degenerate
            tris[t] = c + rng.normal(0.0, 0.3, (3, 3))
            tris[t, 2] = tris[t, 0]
    positions = tris.reshape(-1, 3).astype(np.float32)
    faces = np.arange(3 * n, dtype=np.int32).reshape(n, 3)
    uv = rng.uniform(0.0, 1.0, (3 * n, 2)).astype(np.float32) if rng.random() < 0.8 else None
    mesh = synth.Mesh(positions=positions, faces=faces, uv=uv)
    views = int(rng.integers(1, 4))
    cams = np.zeros((views, 16), np.float32)
    for v in range(views):
        R = _random_rotation(rng)
        cams[v, :12] = np.concatenate([R, rng.normal(0.0, 0.05, (3, 1))], 1).reshape(-1)
        cams[v, 12] = rng.uniform(30.0, 120.0)
    W, H = int(rng.integers(1, 49)), int(rng.integers(1, 49))
    grid_res = tuple(int(g) for g in rng.integers(1, 24, 3)) if rng.random() < 0.3 else (0, 0, 0)
    cells_per_face = float(rng.choice([0.0, 0.5, 2.0, 8.0, 32.0]))
    return mesh, cams, W, H, grid_res, cells_per_face
