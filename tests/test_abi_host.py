"""Host-only checks of the C ABI: the library loads without a GPU, exports
every symbol the header declares, the binding's structs have the header's
layout, and mixrt_validate (pure host code) rejects every bad descriptor."""
import ctypes as C
import os
import re
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
from paper_2312_11841_amd import mixrt, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mixrt.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mixrt_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    declared = _declared_functions()
    assert set(declared) == set(mixrt.EXPORTS)
    L = mixrt.lib()
    for name in declared:
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", mixrt.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (mixrt_\w+)", out))
    assert set(declared) <= exported


LLVM = "/opt/rocm/llvm/bin"


def _code_object_output(obj, tool_args):
    """Runs an LLVM tool on the gfx950 code object of one object file of this
    build (its offload bundle) and returns what the tool printed."""
    with tempfile.TemporaryDirectory() as d:
        fat, co = os.path.join(d, "fat.bin"), os.path.join(d, "co.elf")
        subprocess.run([f"{LLVM}/llvm-objcopy", f"--dump-section=.hip_fatbin={fat}", obj],
                       check=True, capture_output=True)
        subprocess.run([f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o",
                        f"--input={fat}", "--targets=hipv4-amdgcn-amd-amdhsa--gfx950",
                        f"--output={co}"], check=True, capture_output=True)
        return subprocess.run(tool_args + [co], check=True, capture_output=True,
                              text=True).stdout


def _kernel_metadata(obj, field):
    """{kernel: value of an integer metadata field} of the gfx950 code in one
    object file of this build (its offload bundle's kernel metadata)."""
    notes = _code_object_output(obj, [f"{LLVM}/llvm-readelf", "--notes"])
    names = re.findall(r"^\s+\.name:\s+(\S+)", notes, flags=re.M)
    values = [int(v) for v in re.findall(rf"\.{field}:\s+(\d+)", notes)]
    assert len(names) == len(values)
    return dict(zip(names, values))


def _kernel_disassembly(obj):
    """{kernel: [instruction mnemonics with operands]} of the gfx950 code in
    one object file of this build (AMD assembly of the library's own code)."""
    text = _code_object_output(obj, [f"{LLVM}/llvm-objdump", "-d", "--no-show-raw-insn",
                                     "--no-leading-addr"])
    out, cur = {}, None
    for line in text.splitlines():
        m = re.match(r"^<(\S+)>:$", line)
        if m:
            cur = out.setdefault(m.group(1), [])
        elif cur is not None and line.startswith("\t"):
            cur.append(line.split("//")[0].strip())
    return out


def _kernel_private_segments(obj):
    return _kernel_metadata(obj, "private_segment_fixed_size")


@pytest.mark.parametrize("source", ["mixrt_render", "mixrt_stages", "mixrt_raycast",
                                    "mixrt_raster", "microbench"])
def test_kernels_use_no_scratch(source):
    """No kernel of the library has a private (scratch) segment: no register
    spills on the hot path, and no scratch memory the HIP runtime would have
    to allocate at a kernel's first launch (mixrt_render_noalloc allocates
    nothing, and neither does the runtime on its behalf)."""
    from paper_2312_11841_amd import build
    obj = os.path.join(build.OBJ_DIR, source + ".o")
    if not os.path.exists(obj):
        pytest.skip("library objects not built")
    sizes = _kernel_private_segments(obj)
    assert sizes, source
    assert {k: v for k, v in sizes.items() if v} == {}


# The render kernels of the 1280x720 view and the 8-view batch (fp16 grid
# of 2 features, along-ray map, MLP 48-64-64-4) and of the paper's deployed
# grid, with the waves per SIMD their registers allow: 512 VGPRs per lane
# and SIMD, allocated in granules of 8.
HOT_KERNELS = {
    "_ZN5mixrt19render_queue_kernelILi1ELi2ELb1ELi48ELi64ELi2EEE": 3,
    "_ZN5mixrt13render_kernelILi1ELi2ELb1ELi48ELi64ELi2EEE": 3,
    "_ZN5mixrt13render_kernelILi5ELi4ELb1ELi32ELi64ELi2EEE": 2,
}


def test_hot_kernels_keep_their_occupancy():
    """The measured workloads' kernels keep the waves per SIMD their launch
    rules and timings assume (a few more registers in these kernels have
    cost 20% by dropping a wave)."""
    from paper_2312_11841_amd import build
    obj = os.path.join(build.OBJ_DIR, "mixrt_render.o")
    if not os.path.exists(obj):
        pytest.skip("library objects not built")
    vgprs = _kernel_metadata(obj, "vgpr_count")
    for prefix, waves in HOT_KERNELS.items():
        found = [v for k, v in vgprs.items() if k.startswith(prefix)]
        assert len(found) == 1, prefix
        granule = (found[0] + 7) // 8 * 8
        assert 512 // granule >= waves, (prefix, found[0])


@pytest.mark.parametrize("variant", ["timer", "split_nodisp", "split_nohash", "split_nomlp"])
def test_profiling_builds_export_the_same_symbols(variant):
    """The profiling builds (the render kernel compiled with one -D option)
    are drop-in replacements of libmixrt.so for the binding."""
    L = mixrt.lib(variant)
    for name in _declared_functions():
        assert hasattr(L, name), name
    assert L is not mixrt.lib()


def test_microbench_library_exports_every_declared_symbol():
    from paper_2312_11841_amd import microbench
    text = open(os.path.join(ROOT, "include", "mixrt_microbench.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    declared = sorted(set(re.findall(r"\b(mixrt_mb_\w+)\s*\(", text)))
    assert declared
    L = microbench.lib()
    for name in declared:
        assert getattr(L, name).argtypes is not None, name   # bound with a signature
    out = subprocess.run(["nm", "-D", "--defined-only", microbench.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r" T (mixrt_mb_\w+)", out))
    assert set(declared) <= exported


def test_every_header_is_checked():
    assert sorted(os.listdir(os.path.join(ROOT, "include"))) == ["mixrt.h", "mixrt_microbench.h"]


def test_struct_layout_matches_header():
    structs = {"mixrt_create_info": mixrt.CreateInfo, "mixrt_launch_plan": mixrt.LaunchPlan,
               "mixrt_gbuffer": mixrt.GBuffer,
               "mixrt_camera": mixrt.Camera, "mixrt_disp_tex": mixrt.DispTex,
               "mixrt_hash_grid": mixrt.HashGrid, "mixrt_mlp": mixrt.Mlp,
               "mixrt_sampling": mixrt.Sampling, "mixrt_mesh_desc": mixrt.MeshDesc,
               "mixrt_mesh_info": mixrt.MeshInfo}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "mixrt.h"', "int main(void){"]
    for cname, py in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines.append("return 0;}")
    with tempfile.TemporaryDirectory() as d:
        src, exe = os.path.join(d, "l.c"), os.path.join(d, "l")
        open(src, "w").write("\n".join(lines))
        subprocess.run(["gcc", "-I", os.path.dirname(HEADER), src, "-o", exe], check=True)
        rows = subprocess.run([exe], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {}
    for r in rows:
        if r:
            a, b, c = r.split()
            got[(a, b)] = int(c)
    for cname, py in structs.items():
        assert got[(cname, "size")] == C.sizeof(py), cname
        for fname, _ in py._fields_:
            assert got[(cname, fname)] == getattr(py, fname).offset, (cname, fname)


def test_status_strings():
    assert mixrt.status_string(0) == "ok"
    for s in (-1, -2, -3, -4):
        assert mixrt.status_string(s) not in ("ok", "unknown status")
    assert mixrt.status_string(-99) == "unknown status"


# --- validation -----------------------------------------------------------------

FAKE = 0x10000  # an aligned address: validate never dereferences device pointers


class _Desc:
    def __init__(self, cfg=synth.VIEW720P):
        self.cfg = cfg
        self.gbuf = mixrt.GBuffer(cfg.views, cfg.W, cfg.H, FAKE, 0)
        cams = np.zeros((cfg.views, 16), np.float32)
        cams[:, [0, 5, 10]] = 1.0
        cams[:, 12] = 60.0
        self.cams = mixrt.make_cameras(cams)
        self.disp = mixrt.DispTex()
        self.disp.R, self.disp.V = cfg.tex_R, cfg.tex_V
        self.disp.dtype = synth.dtype_code(cfg.tex_dtype)
        self.disp.mode = {"ray": 0, "vec3": 1, "none": 2}[cfg.disp]
        self.disp.data = FAKE
        self.disp.C = cfg.tex_C
        self.disp.sh_degree = cfg.sh_degree
        self.disp.scale = FAKE if cfg.disp == "vec3" else 0
        self.disp.q_scale[:] = [0.01, 0.01]
        self.grid = mixrt.HashGrid(cfg.L, cfg.log2_T, cfg.F, cfg.N_min, cfg.N_max,
                                   synth.dtype_code(cfg.table_dtype), FAKE)
        self.mlp = mixrt.Mlp()
        self.mlp.n_layers = len(cfg.widths) - 1
        for i, w in enumerate(cfg.widths):
            self.mlp.width[i] = w
        self.mlp.view_sh_dim = cfg.view_sh_dim
        self.mlp.data = FAKE
        self.smp = mixrt.Sampling(cfg.K, cfg.delta, cfg.t_term)

    def validate(self):
        return mixrt.validate(self.gbuf, self.cams, self.disp, self.grid, self.mlp, self.smp)


@pytest.mark.parametrize("cfg", list(synth.CONFIGS.values()), ids=lambda c: c.name)
def test_validate_accepts_every_workload(cfg):
    rc, msg = _Desc(cfg).validate()
    assert rc == mixrt.MIXRT_OK, msg


def test_descriptor_makers_refuse_wrong_buffers():
    """make_grid and make_mlp check the tensor behind the pointer they hand to
    the library (dtype, layout, size, on a GPU) before any descriptor exists:
    the library cannot see sizes, so a short or host buffer would be read out
    of bounds on the GPU."""
    torch = pytest.importorskip("torch")
    with pytest.raises(ValueError, match="dtype"):
        mixrt.make_grid(torch.zeros((2, 16, 2), dtype=torch.float64), 4, 8)
    with pytest.raises(ValueError, match="power of two"):
        mixrt.make_grid(torch.zeros((2, 24, 2), dtype=torch.float16), 4, 8)
    with pytest.raises(ValueError, match="3-d"):
        mixrt.make_grid(torch.zeros((32, 2), dtype=torch.float16), 4, 8)
    with pytest.raises(ValueError, match="contiguous"):
        mixrt.make_grid(torch.zeros((2, 2, 16), dtype=torch.float16).transpose(1, 2), 4, 8)
    with pytest.raises(ValueError, match="expected a GPU"):
        mixrt.make_grid(torch.zeros((2, 16, 2), dtype=torch.float16), 4, 8)
    w_ok = 16 * 16 + 16 * 4
    with pytest.raises(ValueError, match="elements"):
        mixrt.make_mlp(torch.zeros(w_ok - 1, dtype=torch.float16), (16, 16, 4), 0)
    with pytest.raises(ValueError, match="dtype"):
        mixrt.make_mlp(torch.zeros(w_ok, dtype=torch.float32), (16, 16, 4), 0)
    with pytest.raises(ValueError, match="contiguous"):
        mixrt.make_mlp(torch.zeros(2 * w_ok, dtype=torch.float16)[::2], (16, 16, 4), 0)
    with pytest.raises(ValueError, match="expected a GPU"):
        mixrt.make_mlp(torch.zeros(w_ok, dtype=torch.float16), (16, 16, 4), 0)
    with pytest.raises(TypeError):
        mixrt.make_mlp(None, (16, 16, 4), 0)
    # the MLP removed has no weights to check
    m = mixrt.make_mlp(None, (16,), 0)
    assert m.n_layers == 0 and m.data is None


def test_validate_accepts_every_random_sweep_config():
    from randcfg import SEEDS, random_config
    for seed in SEEDS:
        cfg = random_config(seed)
        rc, msg = _Desc(cfg).validate()
        assert rc == mixrt.MIXRT_OK, (cfg, msg)


BAD = [
    ("gbuf.views", lambda d: setattr(d.gbuf, "views", 0), mixrt.MIXRT_EINVAL),
    ("gbuf.views max", lambda d: setattr(d.gbuf, "views", 17), mixrt.MIXRT_EINVAL),
    ("gbuf.W", lambda d: setattr(d.gbuf, "W", 0), mixrt.MIXRT_EINVAL),
    ("gbuf.huge", lambda d: (setattr(d.gbuf, "W", 65536), setattr(d.gbuf, "H", 65536)),
     mixrt.MIXRT_EUNSUPPORTED),
    ("gbuf.g0 null", lambda d: setattr(d.gbuf, "g0", 0), mixrt.MIXRT_EINVAL),
    ("gbuf.g0 misaligned", lambda d: setattr(d.gbuf, "g0", FAKE + 4), mixrt.MIXRT_EINVAL),
    ("fov", lambda d: setattr(d.cams[0], "fov_y_deg", 180.0), mixrt.MIXRT_EINVAL),
    ("c2w nan", lambda d: d.cams[0].c2w.__setitem__(3, float("nan")), mixrt.MIXRT_EINVAL),
    ("disp.V", lambda d: setattr(d.disp, "V", 17), mixrt.MIXRT_EUNSUPPORTED),
    ("disp.R", lambda d: setattr(d.disp, "R", 0), mixrt.MIXRT_EINVAL),
    ("disp.dtype", lambda d: setattr(d.disp, "dtype", 3), mixrt.MIXRT_EUNSUPPORTED),
    ("disp.mode", lambda d: setattr(d.disp, "mode", 3), mixrt.MIXRT_EUNSUPPORTED),
    # every degree 0..3 is built, but not with every grid and MLP: Eq. 2 as
    # printed with the 720p workload's 48-64-64-4 MLP has no render kernel
    ("disp.vec3 with an unbuilt MLP", lambda d: (setattr(d.disp, "mode", 1),
                                                 setattr(d.disp, "scale", FAKE),
                                                 setattr(d.disp, "sh_degree", 0)),
     mixrt.MIXRT_EUNSUPPORTED),
    ("disp.vec3 degree 4", lambda d: (setattr(d.disp, "mode", 1), setattr(d.disp, "sh_degree", 4)),
     mixrt.MIXRT_EUNSUPPORTED),
    ("disp.vec3 no scale", lambda d: (setattr(d.disp, "mode", 1), setattr(d.disp, "sh_degree", 2),
                                      setattr(d.disp, "C", 32)), mixrt.MIXRT_EINVAL),
    ("disp.C too small", lambda d: setattr(d.disp, "C", 4), mixrt.MIXRT_EINVAL),
    ("disp.u8 nan", lambda d: (setattr(d.disp, "dtype", 2), d.disp.q_scale.__setitem__(0, float("nan"))),
     mixrt.MIXRT_EINVAL),
    ("disp.data", lambda d: setattr(d.disp, "data", 0), mixrt.MIXRT_EINVAL),
    ("grid.L", lambda d: setattr(d.grid, "L", 33), mixrt.MIXRT_EUNSUPPORTED),
    ("grid.log2_T", lambda d: setattr(d.grid, "log2_T", 27), mixrt.MIXRT_EUNSUPPORTED),
    ("grid.F", lambda d: setattr(d.grid, "F", 3), mixrt.MIXRT_EUNSUPPORTED),
    ("grid.N", lambda d: setattr(d.grid, "N_max", 8), mixrt.MIXRT_EINVAL),
    ("grid.dtype", lambda d: setattr(d.grid, "dtype", 2), mixrt.MIXRT_EUNSUPPORTED),
    ("grid.data", lambda d: setattr(d.grid, "data", 0), mixrt.MIXRT_EINVAL),
    ("mlp.in", lambda d: d.mlp.width.__setitem__(0, 64), mixrt.MIXRT_EINVAL),
    ("mlp.out", lambda d: d.mlp.width.__setitem__(3, 3), mixrt.MIXRT_EINVAL),
    ("mlp.hidden", lambda d: (d.mlp.width.__setitem__(1, 48), d.mlp.width.__setitem__(2, 48)),
     mixrt.MIXRT_EUNSUPPORTED),
    ("mlp.uneven", lambda d: d.mlp.width.__setitem__(2, 32), mixrt.MIXRT_EUNSUPPORTED),
    ("mlp.view", lambda d: setattr(d.mlp, "view_sh_dim", 9), mixrt.MIXRT_EUNSUPPORTED),
    ("mlp.layers", lambda d: setattr(d.mlp, "n_layers", 1), mixrt.MIXRT_EUNSUPPORTED),
    ("mlp.data", lambda d: setattr(d.mlp, "data", 0), mixrt.MIXRT_EINVAL),
    ("K=0", lambda d: setattr(d.smp, "K", 0), mixrt.MIXRT_EUNSUPPORTED),
    ("K=65", lambda d: setattr(d.smp, "K", 65), mixrt.MIXRT_EUNSUPPORTED),
    ("delta", lambda d: setattr(d.smp, "delta", -1.0), mixrt.MIXRT_EINVAL),
    ("t_term", lambda d: setattr(d.smp, "t_term", 1.0), mixrt.MIXRT_EINVAL),
    ("unbuilt variant", lambda d: setattr(d.disp, "dtype", 0), mixrt.MIXRT_EUNSUPPORTED),
    ("no map needs no data", lambda d: (setattr(d.disp, "mode", 2), setattr(d.disp, "data", 0),
                                        setattr(d.disp, "R", 0)), mixrt.MIXRT_OK),
]


@pytest.mark.parametrize("name,mutate,code", BAD, ids=[b[0] for b in BAD])
def test_validate_rejects(name, mutate, code):
    d = _Desc()
    mutate(d)
    rc, msg = d.validate()
    assert rc == code, (rc, msg)
    assert bool(msg) == (code != mixrt.MIXRT_OK)


def test_validate_null_descriptors():
    d = _Desc()
    for field in ("gbuf", "disp", "grid", "mlp", "smp"):
        args = dict(gbuf=d.gbuf, cams=d.cams, disp=d.disp, grid=d.grid, mlp=d.mlp, smp=d.smp)
        args[field] = None
        rc, msg = mixrt.validate(**args)
        assert rc == mixrt.MIXRT_EINVAL and "NULL" in msg


@pytest.mark.parametrize("L,nmin,nmax", [(8, 16, 256), (16, 16, 4096), (16, 16, 8192),
                                         (4, 256, 4096), (1, 32, 32), (32, 2, 1 << 20)])
def test_library_level_table_equals_oracle(L, nmin, nmax):
    g = mixrt.HashGrid(L, 19, 2, nmin, nmax, 1, FAKE)
    assert np.array_equal(mixrt.level_resolutions(g), oracle.level_resolutions(L, nmin, nmax))


def test_level_table_rejects_bad_grid():
    with pytest.raises(mixrt.MixrtError):
        mixrt.level_resolutions(mixrt.HashGrid(0, 19, 2, 16, 256, 1, FAKE))


# --- the geometry stage's grid plan (pure host) ---------------------------------

def _plan_refs_numpy(pos, faces, res, lo, hi):
    """The binning rule restated: a triangle is listed in each cell of its
    bounding box padded by 1/500 cell whose padded box its plane crosses."""
    pos = pos.astype(np.float64)
    lo, hi, res = np.array(lo, np.float64), np.array(hi, np.float64), np.array(res)
    cell = (hi - lo) / res
    pad = cell / 500.0
    half = cell * (0.5 + 1.0 / 500.0)
    total = 0
    for f in faces:
        P = pos[f]
        c0 = np.clip(np.floor((P.min(0) - pad - lo) * res / (hi - lo)).astype(int), 0, res - 1)
        c1 = np.clip(np.floor((P.max(0) + pad - lo) * res / (hi - lo)).astype(int), 0, res - 1)
        if np.all(c0 == c1):
            total += 1
            continue
        n = np.cross(P[1] - P[0], P[2] - P[0])
        reach = np.abs(n) @ half
        g = np.stack(np.meshgrid(*[np.arange(a, b + 1) for a, b in zip(c0, c1)], indexing="ij"), -1)
        ctr = lo + (g.reshape(-1, 3) + 0.5) * cell
        total += int(np.sum(np.abs((ctr - P[0]) @ n) <= reach * (1 + 1e-9)))
    return total


def test_mesh_plan_automatic_grid():
    m = synth.make_mesh(3, room_level=3, n_objects=4, object_level=2, n_boxes=3, box_div=4)
    rc, msg, info = mixrt.mesh_plan(m.positions, m.faces, m.uv)
    assert rc == mixrt.MIXRT_OK, msg
    lo, hi, res = np.array(info["lo"]), np.array(info["hi"]), np.array(info["grid_res"])
    assert np.all(lo < m.positions.min(0)) and np.all(hi > m.positions.max(0))
    cells = np.prod(res)
    assert 0.5 * 8 * len(m.faces) < cells < 2.0 * 8 * len(m.faces)   # about 8 cells per face
    assert info["n_faces"] == len(m.faces)
    assert info["n_refs"] == _plan_refs_numpy(m.positions, m.faces, res, lo, hi)
    assert info["device_bytes"] >= 8 * cells + 48 * info["n_refs"] + 32 * len(m.faces)
    rc, _, dense = mixrt.mesh_plan(m.positions, m.faces, m.uv, cells_per_face=32.0)
    assert np.prod(dense["grid_res"]) > 2 * cells


def test_mesh_plan_explicit_grid_and_flat_mesh():
    pos = np.array([[-1, -1, -2], [3, -1, -2], [-1, 3, -2]], np.float32)
    faces = np.array([[0, 1, 2]], np.int32)
    rc, msg, info = mixrt.mesh_plan(pos, faces, grid_res=(7, 5, 3))
    assert rc == mixrt.MIXRT_OK, msg
    assert info["grid_res"] == (7, 5, 3)
    assert info["hi"][2] > info["lo"][2]                     # a flat mesh gets a thick box
    assert info["n_refs"] == _plan_refs_numpy(pos, faces, (7, 5, 3), info["lo"], info["hi"])
    rc, msg, info = mixrt.mesh_plan(pos, faces, grid_res=(1, 1, 1))
    assert rc == mixrt.MIXRT_OK and info["n_refs"] == 1


MESH_BAD = [
    ("index high", lambda p, f, kw: f.__setitem__((0, 1), len(p)), mixrt.MIXRT_EINVAL),
    ("index negative", lambda p, f, kw: f.__setitem__((0, 2), -1), mixrt.MIXRT_EINVAL),
    ("nan vertex", lambda p, f, kw: p.__setitem__((1, 0), np.nan), mixrt.MIXRT_EINVAL),
    ("partial grid_res", lambda p, f, kw: kw.update(grid_res=(4, 0, 4)), mixrt.MIXRT_EINVAL),
    ("grid axis > 1024", lambda p, f, kw: kw.update(grid_res=(1025, 1, 1)), mixrt.MIXRT_EINVAL),
    ("grid > 2^26 cells", lambda p, f, kw: kw.update(grid_res=(1024, 1024, 65)), mixrt.MIXRT_EINVAL),
    ("cells_per_face < 0", lambda p, f, kw: kw.update(cells_per_face=-1.0), mixrt.MIXRT_EINVAL),
    ("cells_per_face nan", lambda p, f, kw: kw.update(cells_per_face=float("nan")), mixrt.MIXRT_EINVAL),
]


@pytest.mark.parametrize("name,mutate,code", MESH_BAD, ids=[b[0] for b in MESH_BAD])
def test_mesh_plan_rejects(name, mutate, code):
    m = synth.make_mesh(3, room_level=1, n_objects=1, object_level=0, n_boxes=1, box_div=1)
    pos, faces, kw = m.positions.copy(), m.faces.copy(), {}
    mutate(pos, faces, kw)
    rc, msg, info = mixrt.mesh_plan(pos, faces, m.uv, **kw)
    assert rc == code and msg and info is None


def test_mesh_plan_rejects_null_and_tiny():
    rc = mixrt.lib().mixrt_mesh_plan(None, None, None, 0)
    assert rc == mixrt.MIXRT_EINVAL
    d = mixrt.MeshDesc(2, 1, 0, 0, None, (C.c_int32 * 3)(0, 0, 0), 0.0)
    assert mixrt.lib().mixrt_mesh_plan(C.byref(d), None, None, 0) == mixrt.MIXRT_EINVAL
    assert b"n_vertices" in mixrt.lib().mixrt_thread_error()


def test_binding_checks_buffers_it_passes_as_pointers():
    """The binding refuses a buffer the library would reach out of bounds."""
    torch = pytest.importorskip("torch")
    with pytest.raises(ValueError, match="on cpu"):
        mixrt._require(torch.zeros(8), "out", (torch.float32,), 8, 0)
    with pytest.raises(TypeError):
        mixrt._require(np.zeros(8, np.float32), "out", (torch.float32,), 8, 0)


@pytest.mark.parametrize("flags", [8, 1 << 31, mixrt.MIXRT_FLAG_BLOCKS_FULL | mixrt.MIXRT_FLAG_BLOCKS_TWO])
def test_create_rejects_bad_flags_before_touching_a_device(flags):
    """Unknown flag bits, or both block-count flags, are MIXRT_EINVAL (checked
    on the host, so this runs without a GPU)."""
    h = C.c_void_p()
    ci = mixrt.CreateInfo(0, None, flags)
    assert mixrt.lib().mixrt_create(C.byref(h), C.byref(ci)) == mixrt.MIXRT_EINVAL
    assert not h.value
    assert "flag" in mixrt.lib().mixrt_thread_error().decode().lower()


def test_flag_values_match_header():
    text = open(os.path.join(ROOT, "include", "mixrt.h")).read()
    for name in ("MIXRT_FLAG_SYNC_CHECK", "MIXRT_FLAG_BLOCKS_FULL", "MIXRT_FLAG_BLOCKS_TWO"):
        m = re.search(rf"{name}\s*=\s*(\d+)u", text)
        assert m and int(m.group(1)) == getattr(mixrt, name), name


def test_mlp_stage_pipeline_counts_hold():
    """The MLP stage's tile loop waits on hand-counted vmcnt values that hold
    only if every tile issues exactly IN / 8 row loads (into LDS) and one
    output store, and no other vector-memory operation is in flight among
    them.  Checked on the built code of every mlp_kernel instance (one tile
    ahead): the weight loads all come before the first row load, no other
    vector-memory instruction follows it, the two issue sites (the
    prologue's tile and the loop's next tile) hold IN / 8 row loads each,
    there is one store, and every vmcnt wait is within the pipeline's
    depth."""
    from paper_2312_11841_amd import build
    obj = os.path.join(build.OBJ_DIR, "mixrt_stages.o")
    if not os.path.exists(obj):
        pytest.skip("library objects not built")
    kernels = {k: v for k, v in _kernel_disassembly(obj).items() if "mlp_kernel" in k}
    assert len(kernels) >= 6
    vmem = re.compile(r"^(global_|buffer_|flat_|scratch_)")
    for name, ins in kernels.items():
        IN, HID, NHID, DEPTH = map(int, re.search(
            r"mlp_kernelILi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)E", name).groups())
        ch = IN // 8
        ops = [i.split()[0] for i in ins if i]
        loads = [j for j, o in enumerate(ops) if o == "global_load_lds_dwordx4"]
        stores = [j for j, o in enumerate(ops) if o == "global_store_dwordx4"]
        assert DEPTH == 1 and len(loads) == 2 * ch, name
        # each site's loads are straight-line code under the full exec mask:
        # no branch and no exec change between them (a load skipped in some
        # waves would leave the counted waits short)
        for site in (loads[:ch], loads[ch:]):
            between = ins[site[0]:site[-1] + 1]
            assert not [i for i in between if i.startswith("s_cbranch") or "exec" in i], name
        assert len(stores) == 1, name
        others = [ops[j] for j in range(loads[0], len(ops))
                  if vmem.match(ops[j]) and ops[j] not in ("global_load_lds_dwordx4",
                                                           "global_store_dwordx4")]
        assert others == [], (name, others)
        for i in ins:
            m = re.search(r"vmcnt\((\d+)\)", i)
            if m:
                assert int(m.group(1)) <= DEPTH * (ch + 1), (name, i)
