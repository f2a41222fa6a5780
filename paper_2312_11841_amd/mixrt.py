"""Python binding of libmixrt.so (the C ABI in include/mixrt.h).

Argument marshalling only: every step of the rendering path runs in the HIP
kernels behind the C ABI.  PyTorch provides device memory and the stream.
If the library is missing, importing works but every call raises
MixrtUnavailable: there is no CPU fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmixrt.so")

MIXRT_OK = 0
MIXRT_EINVAL = -1
MIXRT_ENOMEM = -2
MIXRT_EDEVICE = -3
MIXRT_EUNSUPPORTED = -4
MIXRT_F32, MIXRT_F16, MIXRT_U8 = 0, 1, 2
MIXRT_DISP_ALONG_RAY, MIXRT_DISP_SH_VEC3, MIXRT_DISP_NONE = 0, 1, 2
_DISP = {"ray": MIXRT_DISP_ALONG_RAY, "vec3": MIXRT_DISP_SH_VEC3, "none": MIXRT_DISP_NONE}
MIXRT_FLAG_SYNC_CHECK = 1
MIXRT_FLAG_BLOCKS_FULL, MIXRT_FLAG_BLOCKS_TWO = 2, 4
_BLOCKS = {None: 0, "full": MIXRT_FLAG_BLOCKS_FULL, "two": MIXRT_FLAG_BLOCKS_TWO}
MAX_VIEWS, MAX_LEVELS, MAX_LAYERS = 16, 32, 8

# Every symbol include/mixrt.h declares.
EXPORTS = (
    "mixrt_create", "mixrt_destroy", "mixrt_sync", "mixrt_validate",
    "mixrt_level_resolutions", "mixrt_render", "mixrt_render_noalloc",
    "mixrt_render_launch_shape",
    "mixrt_debug_phase_cycles", "mixrt_debug_ray_setup",
    "mixrt_debug_hash_encode", "mixrt_debug_mlp", "mixrt_debug_composite",
    "mixrt_mesh_plan", "mixrt_mesh_create", "mixrt_mesh_get_info", "mixrt_mesh_destroy",
    "mixrt_raycast", "mixrt_rasterize",
    "mixrt_status_string", "mixrt_last_error", "mixrt_thread_error",
)
RAY_T_MIN = 1e-4


class MixrtUnavailable(RuntimeError):
    pass


class MixrtError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{status_string(status)} ({status}): {msg}")
        self.status = status


# --- descriptor structs (field order and types as in mixrt.h) ------------------

class CreateInfo(C.Structure):
    _fields_ = [("device", C.c_int32), ("hip_stream", C.c_void_p), ("flags", C.c_uint32),
                ("tile_stripe", C.c_int32), ("early_stop_chunk", C.c_int32),
                ("block_levels", C.c_int32)]


class LaunchPlan(C.Structure):
    _fields_ = [("blocks", C.c_int32), ("tile_stripe", C.c_int32), ("chunk", C.c_int32),
                ("block_from", C.c_int32), ("hash_batch", C.c_int32), ("claims", C.c_int32)]


class GBuffer(C.Structure):
    _fields_ = [("views", C.c_int32), ("W", C.c_int32), ("H", C.c_int32),
                ("g0", C.c_void_p), ("g1", C.c_void_p)]


class Camera(C.Structure):
    _fields_ = [("c2w", C.c_float * 12), ("fov_y_deg", C.c_float), ("bg", C.c_float * 3)]


class DispTex(C.Structure):
    _fields_ = [("R", C.c_int32), ("V", C.c_int32), ("dtype", C.c_int32), ("mode", C.c_int32),
                ("data", C.c_void_p), ("C", C.c_int32), ("sh_degree", C.c_int32),
                ("scale", C.c_void_p), ("q_scale", C.c_float * 2), ("q_offset", C.c_float * 2)]


class HashGrid(C.Structure):
    _fields_ = [("L", C.c_int32), ("log2_T", C.c_int32), ("F", C.c_int32),
                ("N_min", C.c_int32), ("N_max", C.c_int32), ("dtype", C.c_int32),
                ("data", C.c_void_p)]


class Mlp(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("width", C.c_int32 * (MAX_LAYERS + 1)),
                ("view_sh_dim", C.c_int32), ("data", C.c_void_p)]


class Sampling(C.Structure):
    _fields_ = [("K", C.c_int32), ("delta", C.c_float), ("t_term", C.c_float)]


class MeshDesc(C.Structure):
    _fields_ = [("n_vertices", C.c_int64), ("n_faces", C.c_int64), ("positions", C.c_void_p),
                ("faces", C.c_void_p), ("uv", C.c_void_p), ("grid_res", C.c_int32 * 3),
                ("cells_per_face", C.c_float)]


class MeshInfo(C.Structure):
    _fields_ = [("grid_res", C.c_int32 * 3), ("lo", C.c_float * 3), ("hi", C.c_float * 3),
                ("n_faces", C.c_int64), ("n_refs", C.c_int64), ("device_bytes", C.c_int64)]


_libs = {}


def variant_path(variant=None) -> str:
    """Path of libmixrt.so, or of one of its profiling builds ("timer",
    "split_nodisp", "split_nohash", "split_nomlp"; see build.py)."""
    return LIB_PATH if variant is None else os.path.join(_PKG, f"libmixrt_{variant}.so")


def lib(variant=None):
    """Load libmixrt.so (or a profiling build of it), or raise
    MixrtUnavailable (no fallback path exists)."""
    path = variant_path(variant)
    if path not in _libs:
        if not os.path.exists(path):
            raise MixrtUnavailable(
                f"{path} is missing: build it with `python __graft_entry__.py` "
                "or `python paper_2312_11841_amd/build.py`")
        L = C.CDLL(path)
        P, I64 = C.c_void_p, C.c_int64
        sig = {
            "mixrt_create": (C.c_int, [C.POINTER(C.c_void_p), C.POINTER(CreateInfo)]),
            "mixrt_destroy": (C.c_int, [P]),
            "mixrt_sync": (C.c_int, [P]),
            "mixrt_validate": (C.c_int, [C.POINTER(GBuffer), C.POINTER(Camera),
                                         C.POINTER(DispTex), C.POINTER(HashGrid),
                                         C.POINTER(Mlp), C.POINTER(Sampling),
                                         C.c_char_p, C.c_size_t]),
            "mixrt_level_resolutions": (C.c_int, [C.POINTER(HashGrid), P]),
            "mixrt_render": (C.c_int, [P, C.POINTER(GBuffer), C.POINTER(Camera),
                                       C.POINTER(DispTex), C.POINTER(HashGrid), C.POINTER(Mlp),
                                       C.POINTER(Sampling), P]),
            "mixrt_render_noalloc": (C.c_int, [P, C.POINTER(GBuffer), C.POINTER(Camera),
                                               C.POINTER(DispTex), C.POINTER(HashGrid),
                                               C.POINTER(Mlp), C.POINTER(Sampling), P]),
            "mixrt_render_launch_shape": (C.c_int, [P, C.POINTER(GBuffer), C.POINTER(Camera),
                                                    C.POINTER(DispTex), C.POINTER(HashGrid),
                                                    C.POINTER(Mlp), C.POINTER(Sampling),
                                                    C.POINTER(LaunchPlan)]),
            "mixrt_debug_phase_cycles": (C.c_int, [P, P, C.c_int]),
            "mixrt_debug_ray_setup": (C.c_int, [P, C.POINTER(GBuffer), C.POINTER(Camera),
                                                C.POINTER(DispTex), C.POINTER(Sampling), P, P]),
            "mixrt_debug_hash_encode": (C.c_int, [P, C.POINTER(HashGrid), P, I64, P, P, P, P]),
            "mixrt_debug_mlp": (C.c_int, [P, C.POINTER(Mlp), P, I64, P]),
            "mixrt_debug_composite": (C.c_int, [P, P, I64, C.POINTER(Sampling), P, P]),
            "mixrt_mesh_plan": (C.c_int, [C.POINTER(MeshDesc), C.POINTER(MeshInfo), C.c_char_p,
                                          C.c_size_t]),
            "mixrt_mesh_create": (C.c_int, [P, C.POINTER(MeshDesc), C.POINTER(C.c_void_p)]),
            "mixrt_mesh_get_info": (C.c_int, [P, C.POINTER(MeshInfo)]),
            "mixrt_mesh_destroy": (C.c_int, [P]),
            "mixrt_raycast": (C.c_int, [P, P, C.c_int32, C.c_int32, C.c_int32,
                                        C.POINTER(Camera), P, P]),
            "mixrt_rasterize": (C.c_int, [P, P, C.c_int32, C.c_int32, C.c_int32,
                                          C.POINTER(Camera), P, P]),
            "mixrt_status_string": (C.c_char_p, [C.c_int]),
            "mixrt_last_error": (C.c_char_p, [P]),
            "mixrt_thread_error": (C.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _libs[path] = L
    return _libs[path]


def status_string(status: int) -> str:
    return lib().mixrt_status_string(status).decode()


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _require(t, name: str, dtypes, numel: int, device):
    """Check a tensor whose device pointer is handed to the library: of an
    accepted dtype, contiguous, at least numel elements, and on GPU `device`
    (any GPU when device is None).  The library only sees a pointer, so a
    wrong buffer would be read or written out of bounds on the GPU."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if t.dtype not in dtypes:
        raise ValueError(f"{name}: dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: not contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, needs {numel}")
    if t.device.type != "cuda" or (device is not None and t.device.index != device):
        want = "a GPU" if device is None else f"cuda:{device}"
        raise ValueError(f"{name}: on {t.device}, expected {want}")
    return t


# --- descriptors from scene data -------------------------------------------------

_DT = {"float32": MIXRT_F32, "float16": MIXRT_F16, "uint8": MIXRT_U8}


def _dtype_code(t) -> int:
    return _DT[str(t.dtype).replace("torch.", "")]


def make_cameras(cams: np.ndarray):
    cams = np.asarray(cams, np.float32).reshape(-1, 16)
    arr = (Camera * cams.shape[0])()
    for v in range(cams.shape[0]):
        arr[v].c2w[:] = [float(x) for x in cams[v, :12]]
        arr[v].fov_y_deg = float(cams[v, 12])
        arr[v].bg[:] = [float(x) for x in cams[v, 13:16]]
    return arr


def make_sampling(K: int, delta: float, t_term: float) -> Sampling:
    return Sampling(int(K), float(delta), float(t_term))


def make_grid(table, N_min: int, N_max: int) -> HashGrid:
    """Descriptor of a device table [L][T][F] (T a power of two, fp32 or
    fp16, contiguous, on a GPU); it holds a reference to the tensor, so the
    memory it points at lives as long as the descriptor."""
    import torch
    if not isinstance(table, torch.Tensor) or table.dim() != 3:
        raise ValueError("table: expected a 3-d torch.Tensor [L][T][F]")
    L, T, F = (int(n) for n in table.shape)
    if T < 1 or T & (T - 1):
        raise ValueError(f"table: T={T} entries per level is not a power of two")
    _require(table, "table", (torch.float32, torch.float16), L * T * F, None)
    g = HashGrid(L, T.bit_length() - 1, F, int(N_min), int(N_max),
                 _dtype_code(table), _ptr(table))
    g._keep = table
    return g


def mlp_weight_count(widths) -> int:
    """fp16 weights of an MLP with these layer widths (no biases)."""
    return sum(int(a) * int(b) for a, b in zip(widths[:-1], widths[1:]))


def make_mlp(weights, widths, view_sh_dim: int) -> Mlp:
    """Descriptor of device weights (fp16, or their bits as int16; every
    layer's [in][out] matrix concatenated, contiguous, on a GPU); it holds a
    reference to the tensor."""
    import torch
    if len(widths) < 1 or len(widths) > MAX_LAYERS + 1:
        raise ValueError(f"widths: {len(widths)} entries, expected 1..{MAX_LAYERS + 1}")
    n = mlp_weight_count(widths)
    if n > 0 or weights is not None:
        _require(weights, "weights", (torch.float16, torch.int16), n, None)
    m = Mlp()
    m._keep = weights
    m.n_layers = len(widths) - 1
    for i, w in enumerate(widths):
        m.width[i] = int(w)
    m.view_sh_dim = int(view_sh_dim)
    m.data = _ptr(weights)
    return m


@dataclass
class DeviceScene:
    """A scene's arrays in device memory plus the C descriptors that point at
    them.  Keeps the tensors alive as long as the descriptors are used."""

    g0: object
    tex: object
    scale: object
    table: object
    weights: object
    cams: object
    gbuf: GBuffer
    disp: DispTex
    grid: HashGrid
    mlp: Mlp
    smp: Sampling
    rays: int

    @classmethod
    def from_scene(cls, scene, device="cuda"):
        import torch
        cfg = scene.cfg
        g0 = torch.from_numpy(np.ascontiguousarray(scene.g0)).to(device)
        tex = torch.from_numpy(np.ascontiguousarray(scene.tex)).to(device)
        scale = (None if scene.scale is None
                 else torch.from_numpy(np.ascontiguousarray(scene.scale)).to(device))
        table = torch.from_numpy(np.ascontiguousarray(scene.table)).to(device)
        weights = torch.from_numpy(scene.weights_flat.view(np.uint16).astype(np.int16)).to(device)
        gbuf = GBuffer(cfg.views, cfg.W, cfg.rows_kept, _ptr(g0), 0)
        disp = DispTex()
        disp.R, disp.V, disp.dtype = cfg.tex_R, cfg.tex_V, _dtype_code(tex)
        disp.mode = _DISP[cfg.disp]
        disp.data = _ptr(tex)
        disp.C = scene.tex.shape[2]
        disp.sh_degree = cfg.sh_degree
        disp.scale = _ptr(scale)
        disp.q_scale[:] = [float(q) for q in scene.q_scale]
        disp.q_offset[:] = [float(q) for q in scene.q_offset]
        grid = make_grid(table, cfg.N_min, cfg.N_max)
        mlp = make_mlp(weights, cfg.widths, cfg.view_sh_dim)
        smp = make_sampling(cfg.K, cfg.delta, cfg.t_term)
        return cls(g0, tex, scale, table, weights, make_cameras(scene.cams), gbuf, disp, grid,
                   mlp, smp, cfg.rays)

    def check(self, device: int):
        """Every buffer the descriptors point at, against the sizes the
        descriptors declare, before a launch reads it (the library sees only
        pointers)."""
        import torch
        g = self.gbuf
        if g.g0 != _ptr(self.g0):
            raise ValueError("gbuf.g0 does not point at this scene's g0 tensor")
        _require(self.g0, "g0", (torch.float32,), 4 * g.views * g.H * g.W, device)
        d = self.disp
        if d.mode != MIXRT_DISP_NONE:
            tdt = {MIXRT_F32: (torch.float32,), MIXRT_F16: (torch.float16,),
                   MIXRT_U8: (torch.uint8,)}.get(d.dtype, ())
            used = d.V if d.mode == MIXRT_DISP_ALONG_RAY else 3 * (d.sh_degree + 1) ** 2
            chans = d.C if d.C > 0 else used
            if d.data != _ptr(self.tex):
                raise ValueError("disp.data does not point at this scene's texture")
            _require(self.tex, "tex", tdt, d.R * d.R * chans, device)
            if d.mode == MIXRT_DISP_SH_VEC3:
                if self.scale is None or d.scale != _ptr(self.scale):
                    raise ValueError("disp.scale does not point at this scene's scale map")
                _require(self.scale, "scale", tdt, d.R * d.R, device)
        gr = self.grid
        if gr.data != _ptr(self.table):
            raise ValueError("grid.data does not point at this scene's table")
        _require(self.table, "table", (torch.float32, torch.float16),
                 gr.L * (1 << gr.log2_T) * gr.F, device)
        widths = [self.mlp.width[i] for i in range(self.mlp.n_layers + 1)]
        if mlp_weight_count(widths):
            if self.mlp.data != _ptr(self.weights):
                raise ValueError("mlp.data does not point at this scene's weights")
            _require(self.weights, "weights", (torch.float16, torch.int16),
                     mlp_weight_count(widths), device)


# --- meshes (the geometry stage) ---------------------------------------------------

def make_mesh_desc(positions, faces, uv=None, grid_res=(0, 0, 0), cells_per_face=0.0):
    """Descriptor of host arrays; returns (desc, keep) where keep holds the
    contiguous copies the descriptor points to."""
    pos = np.ascontiguousarray(positions, np.float32)
    fc = np.ascontiguousarray(faces, np.int32)
    uvc = None if uv is None else np.ascontiguousarray(uv, np.float32)
    d = MeshDesc(pos.shape[0], fc.shape[0], pos.ctypes.data, fc.ctypes.data,
                 None if uvc is None else uvc.ctypes.data, (C.c_int32 * 3)(*grid_res),
                 float(cells_per_face))
    return d, (pos, fc, uvc)


def _info_dict(info: MeshInfo) -> dict:
    return {"grid_res": tuple(info.grid_res), "lo": tuple(info.lo), "hi": tuple(info.hi),
            "n_faces": info.n_faces, "n_refs": info.n_refs, "device_bytes": info.device_bytes}


def mesh_plan(positions, faces, uv=None, grid_res=(0, 0, 0), cells_per_face=0.0):
    """Pure-host grid plan: (status, message, info dict or None)."""
    d, _keep = make_mesh_desc(positions, faces, uv, grid_res, cells_per_face)
    info = MeshInfo()
    buf = C.create_string_buffer(512)
    rc = lib().mixrt_mesh_plan(C.byref(d), C.byref(info), buf, 512)
    return rc, buf.value.decode(), (_info_dict(info) if rc == MIXRT_OK else None)


class DeviceMesh:
    """A mesh uploaded for the geometry stage (triangle records and the
    ray-casting grid); owns its device memory."""

    def __init__(self, renderer: "Renderer", mesh, grid_res=(0, 0, 0), cells_per_face=0.0):
        d, _keep = make_mesh_desc(mesh.positions, mesh.faces, getattr(mesh, "uv", None),
                                  grid_res, cells_per_face)
        self._L = renderer._L
        h = C.c_void_p()
        renderer._check(self._L.mixrt_mesh_create(renderer._h, C.byref(d), C.byref(h)))
        self._h = h
        info = MeshInfo()
        self._L.mixrt_mesh_get_info(h, C.byref(info))
        self.info = _info_dict(info)

    def close(self):
        if getattr(self, "_h", None):
            self._L.mixrt_mesh_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# --- the library handle ------------------------------------------------------------

class Renderer:
    """One mixrt context bound to a device and a HIP stream."""

    def __init__(self, device: int = 0, stream=None, sync_check: bool = False, blocks=None,
                 tile_stripe: int = 0, early_stop_chunk: int = 0, block_levels: int = 0,
                 variant=None):
        """blocks: None (the library's choice), "full" or "two": the render
        kernel's persistent blocks per CU; tile_stripe: 0 (the library's
        choice), > 0 stripes of that many tiles, < 0 row-major (the order in
        which waves take tiles); early_stop_chunk: 0 (the library's choice),
        < 0 every sample of a ray at once (the tile path), > 0 front to back
        in rounds of that many samples with stopped rays dropped;
        block_levels: 0 (the library's choice), > 0 that many finest levels
        gather x-neighbour corner pairs as 16-byte blocks, < 0 none.  They
        change speed only, never a result.
        variant: None (libmixrt.so) or a profiling build (see lib())."""
        import torch
        self.device = device
        if stream is None:
            stream = torch.cuda.current_stream(device)
        self.stream = stream
        ci = CreateInfo(device, C.c_void_p(int(stream.cuda_stream)),
                        (MIXRT_FLAG_SYNC_CHECK if sync_check else 0) | _BLOCKS[blocks],
                        int(tile_stripe), int(early_stop_chunk), int(block_levels))
        self._L = lib(variant)
        h = C.c_void_p()
        rc = self._L.mixrt_create(C.byref(h), C.byref(ci))
        if rc != MIXRT_OK:
            raise MixrtError(rc, self._L.mixrt_thread_error().decode())
        self._h = h

    def _check(self, rc: int):
        if rc != MIXRT_OK:
            raise MixrtError(rc, self._L.mixrt_last_error(self._h).decode())

    def close(self):
        if getattr(self, "_h", None):
            self._L.mixrt_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def sync(self):
        self._check(self._L.mixrt_sync(self._h))

    # -- the hot path
    def render(self, ds: DeviceScene, out=None):
        import torch
        if out is None:
            out = torch.empty((ds.rays, 4), dtype=torch.float32,
                              device=torch.device("cuda", self.device))
        _require(out, "out", (torch.float32,), 4 * ds.rays, self.device)
        ds.check(self.device)
        self._check(self._L.mixrt_render(self._h, C.byref(ds.gbuf), ds.cams, C.byref(ds.disp),
                                       C.byref(ds.grid), C.byref(ds.mlp), C.byref(ds.smp),
                                       _ptr(out)))
        return out

    def render_noalloc(self, ds: DeviceScene, out):
        """render(ds) through mixrt_render_noalloc: the same frame, with the
        kernels' work counters in the library's fixed per-device array (calls
        that overlap on one device race).  out: the caller's float32 [rays, 4]
        on this device; nothing is allocated."""
        import torch
        _require(out, "out", (torch.float32,), 4 * ds.rays, self.device)
        ds.check(self.device)
        self._check(self._L.mixrt_render_noalloc(self._h, C.byref(ds.gbuf), ds.cams,
                                               C.byref(ds.disp), C.byref(ds.grid),
                                               C.byref(ds.mlp), C.byref(ds.smp), _ptr(out)))
        return out

    def phase_cycles(self, reset: bool = False):
        """The phase-timer build's counters (see mixrt_debug_phase_cycles):
        {"setup", "hash", "mlp", "composite": shader clocks summed over
        waves, "tiles", "waves", "samples": samples evaluated}."""
        out = (C.c_uint64 * 8)()
        self._check(self._L.mixrt_debug_phase_cycles(self._h, out, int(reset)))
        names = ("setup", "hash", "mlp", "composite", "tiles", "waves", "samples")
        return {n: int(out[i]) for i, n in enumerate(names)}

    def launch_shape(self, ds: DeviceScene, chunk: bool = False):
        """(blocks, tile stripe) that render(ds) launches, and with chunk=True
        also its samples per ray per round (0: the tile path)."""
        p = self.launch_plan(ds)
        out = (p["blocks"], p["tile_stripe"], p["chunk"])
        return out if chunk else out[:2]

    def launch_plan(self, ds: DeviceScene) -> dict:
        """The mixrt_launch_plan of render(ds): blocks, tile_stripe, chunk
        (samples per ray per round, 0: the tile path), block_from (first
        level gathered in 16-byte blocks, L: none), hash_batch (hashed
        levels per batch of gathers), claims (1: each wave's last units are
        claimed from the work counters, 0: all in the fixed order)."""
        plan = LaunchPlan()
        self._check(self._L.mixrt_render_launch_shape(
            self._h, C.byref(ds.gbuf), ds.cams, C.byref(ds.disp), C.byref(ds.grid),
            C.byref(ds.mlp), C.byref(ds.smp), C.byref(plan)))
        return {name: int(getattr(plan, name)) for name, _ in LaunchPlan._fields_}

    # -- geometry
    def raycast(self, mesh: DeviceMesh, cams, W: int, H: int, g1: bool = True, out=None):
        """G-buffer of views x H x W pixels by ray casting the mesh's grid:
        (g0, g1) device float [views, H, W, 4] (g1 None unless asked for)."""
        return self._gbuffer(self._L.mixrt_raycast, mesh, cams, W, H, g1, out)

    def rasterize(self, mesh: DeviceMesh, cams, W: int, H: int, g1: bool = True, out=None):
        """The same G-buffer by rasterising the mesh (visibility buffer)."""
        return self._gbuffer(self._L.mixrt_rasterize, mesh, cams, W, H, g1, out)

    def _gbuffer(self, fn, mesh, cams, W, H, g1, out):
        import torch
        cam_arr = cams if isinstance(cams, C.Array) else make_cameras(np.asarray(cams))
        views = len(cam_arr)
        dev = torch.device("cuda", self.device)
        if out is None:
            out = (torch.empty((views, H, W, 4), dtype=torch.float32, device=dev),
                   torch.empty((views, H, W, 4), dtype=torch.float32, device=dev) if g1 else None)
        g0t, g1t = out
        _require(g0t, "out[0]", (torch.float32,), views * H * W * 4, self.device)
        if g1t is not None:
            _require(g1t, "out[1]", (torch.float32,), views * H * W * 4, self.device)
        self._check(fn(self._h, mesh._h, views, W, H, cam_arr, _ptr(g0t), _ptr(g1t)))
        return g0t, g1t

    # -- stage entry points
    def ray_setup(self, ds: DeviceScene):
        import torch
        ds.check(self.device)
        K = ds.smp.K
        x = torch.empty((ds.rays, K, 3), dtype=torch.float32, device=ds.g0.device)
        hit = torch.empty((ds.rays,), dtype=torch.int32, device=ds.g0.device)
        self._check(self._L.mixrt_debug_ray_setup(self._h, C.byref(ds.gbuf), ds.cams,
                                                C.byref(ds.disp), C.byref(ds.smp), _ptr(x),
                                                _ptr(hit)))
        return x, hit

    def hash_encode(self, grid: HashGrid, x, want=("corner", "idx", "w", "feat")):
        import torch
        n = x.shape[0]
        L, F = grid.L, grid.F
        _require(x, "x", (torch.float32,), 3 * n, self.device)
        dev = x.device
        out = {
            "corner": torch.empty((n, L, 3), dtype=torch.int32, device=dev) if "corner" in want else None,
            "idx": torch.empty((n, L, 8), dtype=torch.int32, device=dev) if "idx" in want else None,
            "w": torch.empty((n, L, 8), dtype=torch.float32, device=dev) if "w" in want else None,
            "feat": torch.empty((n, L * F), dtype=torch.float32, device=dev) if "feat" in want else None,
        }
        self._check(self._L.mixrt_debug_hash_encode(
            self._h, C.byref(grid), _ptr(x), n, _ptr(out["corner"]), _ptr(out["idx"]),
            _ptr(out["w"]), _ptr(out["feat"])))
        return out

    def mlp(self, mlp: Mlp, x_f16):
        import torch
        n = x_f16.shape[0]
        _require(x_f16, "x_f16", (torch.float16, torch.int16), n * mlp.width[0], self.device)
        out = torch.empty((n, 4), dtype=torch.float32, device=x_f16.device)
        self._check(self._L.mixrt_debug_mlp(self._h, C.byref(mlp), _ptr(x_f16), n, _ptr(out)))
        return out

    def composite(self, srgb, smp: Sampling, bg):
        import torch
        rays = srgb.shape[0]
        _require(srgb, "srgb", (torch.float32,), rays * smp.K * 4, self.device)
        out = torch.empty((rays, 4), dtype=torch.float32, device=srgb.device)
        bgc = (C.c_float * 3)(*[float(b) for b in bg])
        self._check(self._L.mixrt_debug_composite(self._h, _ptr(srgb), rays, C.byref(smp), bgc,
                                                _ptr(out)))
        return out


def validate(gbuf, cams, disp, grid, mlp, smp):
    """Pure-host descriptor check: returns (status, message)."""
    buf = C.create_string_buffer(512)
    ref = lambda s: None if s is None else C.byref(s)
    rc = lib().mixrt_validate(ref(gbuf), cams, ref(disp), ref(grid), ref(mlp), ref(smp), buf, 512)
    return rc, buf.value.decode()


def level_resolutions(grid: HashGrid) -> np.ndarray:
    out = np.zeros(grid.L, np.int32)
    rc = lib().mixrt_level_resolutions(C.byref(grid), out.ctypes.data)
    if rc != MIXRT_OK:
        raise MixrtError(rc, lib().mixrt_thread_error().decode())
    return out
