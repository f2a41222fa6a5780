"""ctypes front end of the CPU oracle (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path (the HIP library and its binding) never
does.  Every function converts numpy inputs, calls the plain-C oracle in
`mixrt_oracle.c` and returns numpy outputs.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# MIXRT_ORACLE_LIB: load another build of mixrt_oracle.c (the mutation test
# uses it to check that the pins reject planted mistakes).
_LIB_PATH = os.environ.get("MIXRT_ORACLE_LIB", os.path.join(_HERE, "liboracle.so"))
_lib = None

_DT = {np.dtype(np.float32): 0, np.dtype(np.float16): 1, np.dtype(np.uint8): 2}
_DISP = {"ray": 0, "vec3": 1, "none": 2}


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        _lib = C.CDLL(_LIB_PATH)
        _declare(_lib)
    return _lib


def _declare(L):
    P = C.c_void_p
    L.orc_half_to_double.restype = C.c_double
    L.orc_half_to_double.argtypes = [C.c_uint16]
    L.orc_level_resolutions.restype = C.c_int
    L.orc_level_resolutions.argtypes = [C.c_int, C.c_int, C.c_int, P]
    L.orc_sh_real.restype = C.c_double
    L.orc_sh_real.argtypes = [C.c_int, C.c_int, C.c_double, C.c_double, C.c_double]
    L.orc_sh_basis.restype = None
    L.orc_sh_basis.argtypes = [C.c_int, P, P]
    L.orc_camera_ray.restype = None
    L.orc_camera_ray.argtypes = [P, C.c_int, C.c_int, C.c_int, C.c_int, P, P]
    L.orc_tex_bilinear.restype = None
    L.orc_tex_bilinear.argtypes = [P, C.c_int, C.c_int, C.c_int, C.c_double, C.c_double, P]
    L.orc_calibrate.restype = None
    L.orc_calibrate.argtypes = [P, P, P, C.c_int, P]
    L.orc_calibrate_vec3.restype = None
    L.orc_calibrate_vec3.argtypes = [P, P, P, C.c_int, C.c_double, P]
    L.orc_map_bilinear.restype = None
    L.orc_map_bilinear.argtypes = [P, C.c_int, C.c_int, C.c_int, C.c_int, C.c_double,
                                   C.c_double, C.c_double, C.c_double, P]
    L.orc_contract.restype = None
    L.orc_contract.argtypes = [P, P]
    L.orc_hash_level.restype = None
    L.orc_hash_level.argtypes = [P, C.c_int32, C.c_int, C.c_int, C.c_int, P, P, P, P, P]
    L.orc_hash_encode.restype = C.c_int
    L.orc_hash_encode.argtypes = [C.c_int64, P, C.c_int, C.c_int, C.c_int, C.c_int,
                                  C.c_int, C.c_int, P, P, P, P, P]
    L.orc_mlp.restype = C.c_int
    L.orc_mlp.argtypes = [C.c_int64, P, C.c_int, P, P, P]
    L.orc_composite.restype = None
    L.orc_composite.argtypes = [C.c_int64, C.c_int, P, C.c_double, P, P]
    L.orc_render_pixels.restype = C.c_int
    L.orc_render_pixels.argtypes = [P, C.c_int64, P, P, C.c_int]
    L.orc_pixel_samples.restype = C.c_int
    L.orc_pixel_samples.argtypes = [P, C.c_int64, P, P, P, P]
    L.orc_ray_triangle.restype = C.c_int
    L.orc_ray_triangle.argtypes = [P, P, P, P, C.c_int64, P, P, P, P]
    L.orc_ray_mesh.restype = C.c_int64
    L.orc_ray_mesh.argtypes = [P, P, P, P, C.c_int64, P, C.c_double, P, P, P, P, P]
    L.orc_raycast_pixels.restype = C.c_int
    L.orc_raycast_pixels.argtypes = [C.c_int, C.c_int, C.c_int, P, P, P, C.c_int64, P,
                                     C.c_int64, P, P, P, P, P, C.c_int]
    L.orc_max_threads.restype = C.c_int
    L.orc_max_threads.argtypes = []


def _p(a: np.ndarray):
    return C.c_void_p(a.ctypes.data) if a is not None else None


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


class _OrcScene(C.Structure):
    _fields_ = [
        ("views", C.c_int), ("H", C.c_int), ("W", C.c_int),
        ("g0", C.c_void_p), ("cams", C.c_void_p),
        ("tex_R", C.c_int), ("tex_V", C.c_int), ("tex_dtype", C.c_int), ("tex", C.c_void_p),
        ("L", C.c_int), ("log2T", C.c_int), ("F", C.c_int), ("n_min", C.c_int),
        ("n_max", C.c_int), ("table_dtype", C.c_int), ("table", C.c_void_p),
        ("n_layers", C.c_int), ("widths", C.c_void_p), ("view_sh_dim", C.c_int),
        ("weights", C.c_void_p), ("K", C.c_int), ("delta", C.c_double),
        ("disp_mode", C.c_int), ("tex_C", C.c_int), ("sh_degree", C.c_int),
        ("scale", C.c_void_p), ("q_scale", C.c_double * 2), ("q_offset", C.c_double * 2),
    ]


# --- elementary steps ---------------------------------------------------------

def half_to_double(bits) -> np.ndarray:
    bits = np.asarray(bits, dtype=np.uint16).reshape(-1)
    f = lib().orc_half_to_double
    return np.array([f(int(b)) for b in bits], dtype=np.float64)


def level_resolutions(L: int, n_min: int, n_max: int) -> np.ndarray:
    out = np.zeros(L, np.int32)
    if lib().orc_level_resolutions(L, n_min, n_max, _p(out)):
        raise ValueError("bad level schedule")
    return out


def sh_real(l: int, m: int, d) -> float:
    return lib().orc_sh_real(l, m, float(d[0]), float(d[1]), float(d[2]))


def sh_basis(n: int, d) -> np.ndarray:
    d = _c(d, np.float64).reshape(-1, 3)
    out = np.zeros((d.shape[0], n), np.float64)
    for r in range(d.shape[0]):
        row = np.zeros(n, np.float64)
        lib().orc_sh_basis(n, _p(np.ascontiguousarray(d[r])), _p(row))
        out[r] = row
    return out


def camera_ray(cam, W: int, H: int, i: int, j: int):
    cam = _c(cam, np.float32)
    o = np.zeros(3)
    d = np.zeros(3)
    lib().orc_camera_ray(_p(cam), W, H, i, j, _p(o), _p(d))
    return o, d


def tex_bilinear(tex: np.ndarray, u: float, v: float) -> np.ndarray:
    tex = np.ascontiguousarray(tex)
    R, R2, V = tex.shape
    assert R == R2
    out = np.zeros(V)
    lib().orc_tex_bilinear(_p(tex), _DT[tex.dtype], R, V, float(u), float(v), _p(out))
    return out


def map_bilinear(data: np.ndarray, nch: int, u: float, v: float, q_scale=0.0,
                 q_offset=0.0) -> np.ndarray:
    """Bilinear fetch of the first nch of C stored channels ([R][R][C] map)."""
    data = np.ascontiguousarray(data)
    if data.ndim == 2:
        data = data[..., None]
    R, _, Cst = data.shape
    out = np.zeros(nch)
    lib().orc_map_bilinear(_p(data), _DT[data.dtype], R, Cst, nch, float(q_scale),
                           float(q_offset), float(u), float(v), _p(out))
    return out


def calibrate_vec3(p, d, m, nb: int, ms: float) -> np.ndarray:
    p, d, m = _c(p, np.float64), _c(d, np.float64), _c(m, np.float64)
    out = np.zeros(3)
    lib().orc_calibrate_vec3(_p(p), _p(d), _p(m), nb, float(ms), _p(out))
    return out


def calibrate(p, d, m) -> np.ndarray:
    p, d, m = _c(p, np.float64), _c(d, np.float64), _c(m, np.float64)
    out = np.zeros(3)
    lib().orc_calibrate(_p(p), _p(d), _p(m), m.size, _p(out))
    return out


def contract(q) -> np.ndarray:
    q = _c(q, np.float64)
    out = np.zeros(3)
    lib().orc_contract(_p(q), _p(out))
    return out


def hash_encode(x: np.ndarray, table: np.ndarray, n_min: int, n_max: int):
    """x [n,3] fp32 in [0,1]; table [L,T,F] f32/f16.  Returns corner [n,L,3],
    idx [n,L,8], w [n,L,8] and feat [n,L*F]."""
    x = _c(x, np.float32).reshape(-1, 3)
    table = np.ascontiguousarray(table)
    L, T, F = table.shape
    n = x.shape[0]
    corner = np.zeros((n, L, 3), np.int32)
    idx = np.zeros((n, L, 8), np.uint32)
    w = np.zeros((n, L, 8), np.float64)
    feat = np.zeros((n, L * F), np.float64)
    rc = lib().orc_hash_encode(n, _p(x), L, n_min, n_max, int(T).bit_length() - 1, F,
                               _DT[table.dtype], _p(table), _p(corner), _p(idx), _p(w),
                               _p(feat))
    if rc:
        raise ValueError("hash_encode: bad arguments")
    return corner, idx, w, feat


def mlp(inp: np.ndarray, weights) -> np.ndarray:
    """inp [n, w0] (double); weights: list of [in,out] fp16 arrays (empty: the
    MLP removed, inputs summed per component mod 4)."""
    inp = _c(inp, np.float64)
    if not weights:
        widths = np.array([inp.shape[1]], np.int32)
        out = np.zeros((inp.shape[0], 4))
        if lib().orc_mlp(inp.shape[0], _p(inp), 0, _p(widths), None, _p(out)):
            raise ValueError("mlp: bad arguments")
        return out
    widths = np.array([weights[0].shape[0]] + [w.shape[1] for w in weights], np.int32)
    flat = np.concatenate([np.asarray(w, np.float16).reshape(-1) for w in weights])
    bits = flat.view(np.uint16).copy()
    n = inp.shape[0]
    out = np.zeros((n, 4))
    if lib().orc_mlp(n, _p(inp), len(weights), _p(widths), _p(bits), _p(out)):
        raise ValueError("mlp: bad arguments")
    return out


def composite(srgb: np.ndarray, delta: float, bg) -> np.ndarray:
    """srgb [rays,K,4]; bg [rays,3] or [3]."""
    srgb = _c(srgb, np.float64)
    rays, K, _ = srgb.shape
    bg = np.broadcast_to(np.asarray(bg, np.float64), (rays, 3)).copy()
    out = np.zeros((rays, 4))
    lib().orc_composite(rays, K, _p(srgb), float(delta), _p(bg), _p(out))
    return out


# --- the coarse-mesh hit (the G-buffer) ------------------------------------------

def ray_triangle(o, d, positions, faces, f: int):
    """fp64 Moller-Trumbore against triangle f: (t, b1, b2, cos) or None."""
    o, d = _c(o, np.float64), _c(d, np.float64)
    pos, fc = _c(positions, np.float32), _c(faces, np.int32)
    out = np.zeros(4)
    ok = lib().orc_ray_triangle(_p(o), _p(d), _p(pos), _p(fc), f, _p(out[0:]), _p(out[1:]),
                                _p(out[2:]), _p(out[3:]))
    return tuple(out) if ok else None


def ray_mesh(o, d, positions, faces, uv=None, t_min: float = 1e-4):
    """Closest hit over all triangles: dict(tri, t, bary, uv, normal, ambiguous)."""
    o, d = _c(o, np.float64), _c(d, np.float64)
    pos, fc = _c(positions, np.float32), _c(faces, np.int32)
    uvc = None if uv is None else _c(uv, np.float32)
    t, bary, uvo, n = np.zeros(1), np.zeros(2), np.zeros(2), np.zeros(3)
    amb = C.c_int(0)
    f = lib().orc_ray_mesh(_p(o), _p(d), _p(pos), _p(fc), fc.shape[0], _p(uvc), t_min, _p(t),
                           _p(bary), _p(uvo), _p(n), C.byref(amb))
    return {"tri": int(f), "t": float(t[0]), "bary": bary, "uv": uvo, "normal": n,
            "ambiguous": bool(amb.value)}


def raycast_pixels(cams, W: int, H: int, mesh, pix, threads: int = 1):
    """The G-buffer of flat pixel indices (view-major) by brute force:
    (g0 [n,4] f64 (t, u, v, 0) with t = -1 for a miss, normal [n,3], tri [n],
    ambiguous [n] bool)."""
    cams = _c(cams, np.float32).reshape(-1, 16)
    pos, fc = _c(mesh.positions, np.float32), _c(mesh.faces, np.int32)
    uv = None if mesh.uv is None else _c(mesh.uv, np.float32)   # NULL: no texture coordinates
    pix = _c(pix, np.int64).reshape(-1)
    g0, n = np.zeros((pix.size, 4)), np.zeros((pix.size, 3))
    tri, amb = np.zeros(pix.size, np.int64), np.zeros(pix.size, np.int32)
    lib().orc_raycast_pixels(cams.shape[0], H, W, _p(cams), _p(pos), _p(fc), fc.shape[0],
                             _p(uv), pix.size, _p(pix), _p(g0), _p(n), _p(tri), _p(amb),
                             threads)
    return g0, n, tri, amb.astype(bool)


# --- the whole path -------------------------------------------------------------

class OracleScene:
    """Binds a synth.Scene to the oracle's scene descriptor."""

    def __init__(self, scene):
        cfg = scene.cfg
        self.scene = scene
        self.K = cfg.K
        self._keep = []
        g0 = np.ascontiguousarray(scene.g0, np.float32)
        cams = np.ascontiguousarray(scene.cams, np.float32)
        widths = np.array(cfg.widths, np.int32)
        wbits = (scene.weights_flat.view(np.uint16).copy() if scene.weights
                 else np.zeros(1, np.uint16))
        self._keep += [g0, cams, widths, wbits, scene.tex, scene.table]
        s = _OrcScene()
        s.views, s.H, s.W = cfg.views, cfg.rows_kept, cfg.W
        s.g0, s.cams = g0.ctypes.data, cams.ctypes.data
        s.tex_R, s.tex_V = cfg.tex_R, cfg.tex_V
        s.tex_dtype = _DT[scene.tex.dtype]
        s.tex = scene.tex.ctypes.data
        s.L, s.log2T, s.F = cfg.L, cfg.log2_T, cfg.F
        s.n_min, s.n_max = cfg.N_min, cfg.N_max
        s.table_dtype = _DT[scene.table.dtype]
        s.table = scene.table.ctypes.data
        s.n_layers = len(cfg.widths) - 1
        s.widths = widths.ctypes.data
        s.view_sh_dim = cfg.view_sh_dim
        s.weights = wbits.ctypes.data
        s.K, s.delta = cfg.K, float(cfg.delta)
        s.disp_mode = _DISP[cfg.disp]
        s.tex_C = scene.tex.shape[2]
        s.sh_degree = cfg.sh_degree
        if scene.scale is not None:
            self._keep.append(scene.scale)
            s.scale = scene.scale.ctypes.data
        s.q_scale[:] = [float(q) for q in scene.q_scale]
        s.q_offset[:] = [float(q) for q in scene.q_offset]
        self.desc = s

    def render_pixels(self, pix, threads: int = 1) -> np.ndarray:
        pix = _c(pix, np.int64).reshape(-1)
        out = np.zeros((pix.size, 4))
        rc = lib().orc_render_pixels(C.byref(self.desc), pix.size, _p(pix), _p(out), threads)
        if rc:
            raise ValueError("render_pixels: bad scene")
        return out

    def pixel_samples(self, pix):
        pix = _c(pix, np.int64).reshape(-1)
        x = np.zeros((pix.size, self.K, 3), np.float32)
        xd = np.zeros((pix.size, self.K, 3), np.float64)
        hit = np.zeros(pix.size, np.int32)
        lib().orc_pixel_samples(C.byref(self.desc), pix.size, _p(pix), _p(x), _p(xd), _p(hit))
        return x, xd, hit


def max_threads() -> int:
    return lib().orc_max_threads()
