"""GPU parity of the geometry stage (the coarse-mesh hit per pixel, Fig. 2
step 1, by mixrt_raycast and by mixrt_rasterize) against the oracle's
brute-force fp64 ray casting, and of the whole pipeline on mesh-driven
workloads.

Bars, for pixels the oracle does not flag as ambiguous (a hit within the
rounding reach of an edge, another triangle within it in depth, or a near
miss; grazing rays widen that reach):
  - triangle index and hit/miss: bit-exact;
  - t: |dt| <= (1e-5 t + 1e-6 D S) / |cos|.  The fp32 ray direction carries
    about 2e-7 relative error, which moves the hit by t 2e-7 / |cos| along
    the ray; the fp32 Moller-Trumbore solve forms t from products of
    vectors of length ~D (D = the farthest vertex's distance from the
    camera), so it adds a few ulp of D times the condition number S / |cos|
    (S = L_max^2 / (2 area), about 1 / sin of the smallest corner angle);
    both coefficients leave a 10x margin or more;
  - uv: |duv| <= spread (1e-4 + 1e-6 D S / L_max) / |cos| + 1e-6, spread =
    the largest uv difference between the triangle's corners (the
    barycentric error of the moved hit point, ~ulp(D) S / L_max, times the
    uv range it scales); exactly 0 for a mesh without uv;
  - normal: 1e-4 absolute (edges are differenced in fp32 on the GPU).
Ambiguous pixels: the GPU's triangle must be one the oracle also finds hit or
nearly hit, at the same distance, no farther than the nearest hit's reach;
a GPU miss must be a pixel the oracle marks ambiguous.  At most 1% of the
pixels may be ambiguous.
"""
import numpy as np
import pytest

import oracle
from paper_2312_11841_amd import mixrt, synth
import meshbars

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

FRAME_TOL = 2e-3


@pytest.fixture(scope="module")
def R():
    r = mixrt.Renderer(0, sync_check=True)
    yield r
    r.close()


def say(*a):
    print(*a, flush=True)


METHODS = ["raycast", "rasterize"]


def gbuffer(R, method, dm, cams, W, H, g1=True, out=None):
    return getattr(R, method)(dm, cams, W, H, g1=g1, out=out)


def _pixel_dirs(cams, W, H):
    """Unit ray directions of every pixel (view-major), in fp64 from the
    camera rows: the rays of the pixel-ray formula, vectorised."""
    out = []
    j, i = np.mgrid[0:H, 0:W]
    for c in np.asarray(cams, np.float64).reshape(-1, 16):
        f = 0.5 * H / np.tan(np.deg2rad(c[12]) / 2)
        dc = np.stack([(i + 0.5 - W / 2) / f, -(j + 0.5 - H / 2) / f, -np.ones_like(i, float)], -1)
        d = dc.reshape(-1, 3) @ c[:12].reshape(3, 4)[:, :3].T
        out.append(d / np.linalg.norm(d, axis=1, keepdims=True))
    return np.concatenate(out)


def _cams(cam_rows):
    return np.asarray(cam_rows, np.float32).reshape(-1, 16)


def _view_cams(n, fov=60.0, bg=(0.2, 0.4, 0.6)):
    """n poses inside the room, clear of every object."""
    rows = []
    for v in range(n):
        R = synth._rot_y(360.0 * v / n + 15.0) @ synth._rot_x(-5.0 + 7.0 * v)
        o = np.array([0.3 * np.cos(v), 0.2, -0.1 + 0.2 * np.sin(v)])
        row = np.zeros(16, np.float32)
        row[:12] = np.concatenate([R, o[:, None]], 1).reshape(-1)
        row[12], row[13:16] = fov, bg
        rows.append(row)
    return np.stack(rows)


def _check_gbuffer(mesh, cams, W, H, g0, g1, pix, label, max_amb=0.01):
    """Compare the GPU G-buffer (numpy [views*H*W, 4] each) with the oracle at
    the flat pixel indices pix."""
    ref_g0, ref_n, ref_tri, amb = oracle.raycast_pixels(cams, W, H, mesh, pix,
                                                         threads=oracle.max_threads())
    got0, got1 = g0[pix], g1[pix]
    gid = got1[:, 3].view(np.int32)
    ok = ~amb
    say(f"  {label}: {pix.size} px, ambiguous {amb.mean():.4%}, misses {(ref_tri < 0).mean():.2%}")
    assert amb.mean() <= max_amb
    # unique answers
    assert np.array_equal(gid[ok], ref_tri[ok])
    hit = ok & (ref_tri >= 0)
    miss = ok & (ref_tri < 0)
    assert np.all(got0[miss] == np.array([-1, 0, 0, 0], np.float32))
    assert np.all(got1[miss, :3] == 0)
    if hit.any():
        hw = H * W
        view, rem = np.divmod(pix[hit], hw)
        j, i = np.divmod(rem, W)
        d = np.array([oracle.camera_ray(cams[v], W, H, ii, jj)[1]
                      for v, ii, jj in zip(view, i, j)])
        cos = np.abs(np.einsum("ij,ij->i", d, ref_n[hit]))
        # conditioning of the fp32 solve (tests/meshbars.py): the vertices'
        # distance from the camera, the longest edge and the triangle's shape
        origin = np.asarray(cams, np.float64).reshape(-1, 16)[view][:, [3, 7, 11]]
        dist, l_max, shape = meshbars.conditioning(mesh.positions, mesh.faces, ref_tri[hit],
                                                   origin)
        t_ref = ref_g0[hit, 0]
        dt = np.abs(got0[hit, 0] - t_ref)
        tb = meshbars.t_bar(t_ref, dist, shape, cos)
        assert np.all(dt <= tb), ((dt / tb).max(), (dt / t_ref).max())
        terr = dt / t_ref
        uerr = np.abs(got0[hit, 1:3] - ref_g0[hit, 1:3]).max(1)
        if mesh.uv is None:
            assert np.all(got0[hit, 1:3] == 0)
        else:
            corners = mesh.uv.astype(np.float64)[mesh.faces[ref_tri[hit]]]      # [n, 3, 2]
            spread = (corners.max(1) - corners.min(1)).max(1)
            ub = meshbars.uv_bar(spread, dist, shape, l_max, cos)
            assert np.all(uerr <= ub), ((uerr / ub).max(), uerr.max())
        say(f"  largest share of the bars used: t {(dt / tb).max():.3f}"
            + ("" if mesh.uv is None else f", uv {(uerr / ub).max():.3f}"))
        assert np.all(got0[hit, 3] == 0)
        nerr = np.abs(got1[hit, :3] - ref_n[hit]).max()
        assert nerr <= 1e-4, nerr
        say(f"  max rel t err {terr.max():.2e}, uv err {uerr.max():.2e}, normal err {nerr:.2e}")
    # ambiguous pixels: the GPU's answer must be a valid one
    hw = H * W
    for q in np.nonzero(amb)[0]:
        p = int(pix[q])
        view, rem = divmod(p, hw)
        jj, ii = divmod(rem, W)
        o, d = oracle.camera_ray(cams[view], W, H, ii, jj)
        if gid[q] < 0:
            continue            # a near miss or a crack between near-edge hits
        sol = oracle.ray_triangle(o, d, mesh.positions, mesh.faces, int(gid[q]))
        assert sol is not None
        t, b1, b2, c = sol
        g = max(1.0, 0.1 / max(abs(c), 1e-12))
        P = mesh.positions.astype(np.float64)[mesh.faces[int(gid[q])]]
        dist = np.linalg.norm(P - o, axis=1).max()
        e = np.stack([P[1] - P[0], P[2] - P[1], P[0] - P[2]])
        shape = (np.linalg.norm(e, axis=1).max() ** 2
                 / np.linalg.norm(np.cross(e[0], -e[2])))
        assert min(b1, b2, 1 - b1 - b2) > -4e-4 * g
        assert abs(got0[q, 0] - t) <= (meshbars.T_REL * t + meshbars.T_COND * dist * shape) * g
        if ref_tri[q] >= 0:
            assert t <= ref_g0[q, 0] * (1 + 2e-4 * g)


# --------------------------------------------------------------------------
# The ray-casting kernel alone
# --------------------------------------------------------------------------

@pytest.mark.parametrize("method", METHODS)
def test_gbuffer_small_mesh_every_pixel(R, method):
    sc = synth.make_scene(synth.TINY64_MESH)
    cfg = sc.cfg
    say(method, cfg.name, len(sc.mesh.faces), "faces")
    dm = mixrt.DeviceMesh(R, sc.mesh)
    g0, g1 = gbuffer(R, method, dm, sc.cams, cfg.W, cfg.H)
    R.sync()
    pix = np.arange(cfg.rays)
    _check_gbuffer(sc.mesh, _cams(sc.cams), cfg.W, cfg.H, g0.cpu().numpy().reshape(-1, 4),
                   g1.cpu().numpy().reshape(-1, 4), pix, cfg.name)
    dm.close()


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("W,H,views", [(37, 23, 3), (16, 16, 1), (1, 1, 2), (200, 9, 1)])
def test_gbuffer_ragged_shapes_and_views(R, method, W, H, views):
    say(method, "ragged", W, H, views)
    mesh = synth.make_mesh(9, room_level=3, n_objects=5, object_level=2, n_boxes=3, box_div=2)
    cams = _view_cams(views, fov=75.0)
    dm = mixrt.DeviceMesh(R, mesh)
    g0, g1 = gbuffer(R, method, dm, cams, W, H)
    R.sync()
    _check_gbuffer(mesh, cams, W, H, g0.cpu().numpy().reshape(-1, 4),
                   g1.cpu().numpy().reshape(-1, 4), np.arange(views * H * W), f"{W}x{H}x{views}")


@pytest.mark.parametrize("method", METHODS)
def test_gbuffer_wall_with_misses(R, method):
    """A square wall in front of the camera: the border pixels miss."""
    pos = np.array([[-2, -2, -5], [2, -2, -5], [2, 2, -5], [-2, 2, -5]], np.float32)
    faces = np.array([[0, 1, 2], [0, 2, 3]], np.int32)
    uv = ((pos[:, :2] + 2) / 4).astype(np.float32)
    mesh = synth.Mesh(positions=pos, faces=faces, uv=uv)
    cam = np.zeros((1, 16), np.float32)
    # off centre, so that the wall's diagonal edge does not run through a
    # line of pixel centres
    cam[0, :12] = np.concatenate([np.eye(3), np.array([[0.0131], [-0.0217], [0.0]])],
                                 1).reshape(-1)
    cam[0, 12] = 60.0
    W, H = 48, 40
    dm = mixrt.DeviceMesh(R, mesh)
    g0, g1 = gbuffer(R, method, dm, cam, W, H)
    R.sync()
    g0n, g1n = g0.cpu().numpy().reshape(-1, 4), g1.cpu().numpy().reshape(-1, 4)
    assert (g0n[:, 0] == -1).any() and (g0n[:, 0] > 0).any()
    _check_gbuffer(mesh, cam, W, H, g0n, g1n, np.arange(W * H), "wall")


@pytest.mark.parametrize("method", METHODS)
def test_gbuffer_all_miss_and_no_uv(R, method):
    """Looking away from a single triangle: every pixel misses (id -1)."""
    pos = np.array([[-1, -1, 2], [1, -1, 2], [0, 1, 2]], np.float32)
    mesh = synth.Mesh(positions=pos, faces=np.array([[0, 1, 2]], np.int32), uv=None)
    cam = np.zeros((1, 16), np.float32)
    cam[0, :12] = np.concatenate([np.eye(3), np.zeros((3, 1))], 1).reshape(-1)
    cam[0, 12] = 50.0
    dm = mixrt.DeviceMesh(R, mesh)
    g0, g1 = gbuffer(R, method, dm, cam, 20, 10)
    R.sync()
    assert torch.all(g0[..., 0] == -1) and torch.all(g0[..., 1:] == 0)
    assert np.all(g1.cpu().numpy()[..., 3].view(np.int32) == -1)
    # turned round (c2w rotation of 180 degrees about y) it sees the triangle; uv is 0
    cam[0, :12] = np.concatenate([synth._rot_y(180.0), np.zeros((3, 1))], 1).reshape(-1)
    g0, g1 = gbuffer(R, method, dm, cam, 20, 10)
    R.sync()
    hit = g0[..., 0] > 0
    assert hit.any() and torch.all(g0[hit][:, 1:] == 0)


def test_raycast_grid_resolution_does_not_change_the_answer(R):
    """The grid only prunes: a 1x1x1 grid (every triangle tested), a coarse
    and a dense one give bitwise the same G-buffer on unambiguous pixels."""
    mesh = synth.make_mesh(10, room_level=4, n_objects=8, object_level=2, n_boxes=4, box_div=3)
    cams = _view_cams(2)
    W, H = 96, 64
    outs = []
    for res, cpf in (((1, 1, 1), 0.0), ((5, 4, 3), 0.0), ((0, 0, 0), 0.0), ((0, 0, 0), 16.0)):
        dm = mixrt.DeviceMesh(R, mesh, grid_res=res, cells_per_face=cpf)
        say("  grid", dm.info["grid_res"], "refs", dm.info["n_refs"])
        g0, g1 = R.raycast(dm, cams, W, H)
        R.sync()
        outs.append((g0.cpu().numpy().reshape(-1, 4), g1.cpu().numpy().reshape(-1, 4)))
        dm.close()
    pix = np.arange(2 * W * H)
    _, _, _, amb = oracle.raycast_pixels(cams, W, H, mesh, pix, threads=oracle.max_threads())
    for g0n, g1n in outs[1:]:
        assert np.array_equal(g0n[~amb], outs[0][0][~amb])
        assert np.array_equal(g1n[~amb], outs[0][1][~amb])


@pytest.mark.parametrize("method", METHODS)
def test_gbuffer_500k_mesh_sampled(R, method):
    """The 499,712-triangle mesh at 1280x720, in the launch the benchmark
    times, against the oracle on sampled pixels (and the image corners)."""
    cfg = synth.MESH720P
    sc = synth.make_scene(cfg)
    say(method, cfg.name, len(sc.mesh.faces), "faces")
    dm = mixrt.DeviceMesh(R, sc.mesh)
    say("  grid", dm.info)
    g0, g1 = gbuffer(R, method, dm, sc.cams, cfg.W, cfg.H)
    R.sync()
    rng = np.random.default_rng(21)
    pix = np.unique(np.concatenate([rng.choice(cfg.rays, 1200, replace=False),
                                    [0, cfg.W - 1, cfg.rays - cfg.W, cfg.rays - 1]]))
    _check_gbuffer(sc.mesh, _cams(sc.cams), cfg.W, cfg.H, g0.cpu().numpy().reshape(-1, 4),
                   g1.cpu().numpy().reshape(-1, 4), pix, cfg.name)
    a = g0.clone()
    gbuffer(R, method, dm, sc.cams, cfg.W, cfg.H, out=(g0, g1))
    R.sync()
    assert torch.equal(a, g0)                       # deterministic


def test_rasterize_equals_raycast_on_the_500k_mesh(R):
    """Both routes take the fp32 closest hit of the same rays: the same
    triangle except where two hits lie within rounding of each other (the
    rasteriser orders hits with the unnormalised ray direction), and the
    same hit up to fp32 rounding."""
    cfg = synth.MESH720P
    sc = synth.make_scene(cfg)
    dm = mixrt.DeviceMesh(R, sc.mesh)
    cams = _view_cams(3)
    a0, a1 = R.raycast(dm, cams, cfg.W, cfg.H)
    b0, b1 = R.rasterize(dm, cams, cfg.W, cfg.H)
    R.sync()
    ida = a1.cpu().numpy()[..., 3].view(np.int32)
    idb = b1.cpu().numpy()[..., 3].view(np.int32)
    diff = (ida != idb).mean()
    say(f"  triangle differs on {diff:.2e} of {ida.size} px")
    assert diff <= 1e-4
    # where the two routes pick different triangles, both answers must lie
    # within fp32 rounding of each other: the oracle flags such pixels
    # ambiguous
    odd = np.nonzero((ida != idb).reshape(-1))[0]
    if odd.size:
        _, _, _, amb = oracle.raycast_pixels(cams, cfg.W, cfg.H, sc.mesh, odd,
                                             threads=oracle.max_threads())
        assert np.all(amb), odd[~amb]
    # t: the same formula on the same fp32 inputs, compiled in two kernels
    # (multiply-adds may contract differently); grazing hits amplify that
    # like any fp32 rounding, so the oracle bar's 1/|cos| factor applies
    same = ida == idb
    ta = a0.cpu().numpy()[..., 0][same].astype(np.float64)
    tb = b0.cpu().numpy()[..., 0][same].astype(np.float64)
    rel = np.abs(ta - tb) / ta
    nrm = a1.cpu().numpy()[..., :3].reshape(-1, 3)[same.reshape(-1)]
    dirs = _pixel_dirs(cams, cfg.W, cfg.H)[same.reshape(-1)]
    cos = np.maximum(np.abs(np.einsum("ij,ij->i", dirs, nrm)), 1e-3)
    say(f"  t: max rel diff {rel.max():.2e}, p99.99 {np.percentile(rel, 99.99):.2e}")
    assert np.all(rel <= 1e-5 / cos)


@pytest.mark.parametrize("method", METHODS)
def test_gbuffer_geometry_around_and_behind_the_camera(R, method):
    """Large triangles that surround the camera, straddle its plane and lie
    behind it (the rasteriser clips them), and a small one a hair beyond the
    minimum hit distance."""
    rng = np.random.default_rng(23)
    big = rng.uniform(-3, 3, (40, 3, 3)).astype(np.float32)
    near = np.array([[[-1e-3, -1e-3, -2.5e-4], [1e-3, -1e-3, -2.5e-4], [0.0, 1e-3, -2.5e-4]]],
                    np.float32)
    tris = np.concatenate([big, near])
    mesh = synth.Mesh(positions=tris.reshape(-1, 3),
                      faces=np.arange(3 * len(tris), dtype=np.int32).reshape(-1, 3),
                      uv=rng.uniform(0, 1, (3 * len(tris), 2)).astype(np.float32))
    cams = np.zeros((2, 16), np.float32)
    cams[0, :12] = np.concatenate([np.eye(3), np.zeros((3, 1))], 1).reshape(-1)
    cams[1, :12] = np.concatenate([synth._rot_y(70.0) @ synth._rot_x(20.0),
                                   np.array([[0.3], [-0.2], [0.5]])], 1).reshape(-1)
    cams[:, 12] = (90.0, 120.0)
    W, H = 64, 48
    dm = mixrt.DeviceMesh(R, mesh)
    g0, g1 = gbuffer(R, method, dm, cams, W, H)
    R.sync()
    _check_gbuffer(mesh, cams, W, H, g0.cpu().numpy().reshape(-1, 4),
                   g1.cpu().numpy().reshape(-1, 4), np.arange(2 * W * H), "around", max_amb=0.05)


def test_rasterize_rejects(R):
    mesh = synth.make_mesh(3, room_level=1, n_objects=1, object_level=0, n_boxes=1, box_div=1)
    dm = mixrt.DeviceMesh(R, mesh)
    cams = mixrt.make_cameras(_view_cams(1))
    buf = torch.empty(8 * 8 * 4, dtype=torch.float32, device="cuda")
    lib = mixrt.lib()
    assert lib.mixrt_rasterize(R._h, dm._h, 1, 8192, 8192, cams, buf.data_ptr(),
                               None) == mixrt.MIXRT_EUNSUPPORTED
    assert lib.mixrt_rasterize(R._h, dm._h, 0, 8, 8, cams, buf.data_ptr(), None) == mixrt.MIXRT_EINVAL
    assert lib.mixrt_rasterize(R._h, dm._h, 1, 8, 8, cams, buf.data_ptr() + 8,
                               None) == mixrt.MIXRT_EINVAL


def test_raycast_rejects(R):
    mesh = synth.make_mesh(3, room_level=1, n_objects=1, object_level=0, n_boxes=1, box_div=1)
    dm = mixrt.DeviceMesh(R, mesh)
    cam = _view_cams(1)
    buf = torch.empty(8 * 8 * 4 + 1, dtype=torch.float32, device="cuda")
    lib = mixrt.lib()
    cams = mixrt.make_cameras(cam)
    assert lib.mixrt_raycast(R._h, dm._h, 0, 8, 8, cams, buf.data_ptr(), None) == mixrt.MIXRT_EINVAL
    assert lib.mixrt_raycast(R._h, dm._h, 1, 8, 0, cams, buf.data_ptr(), None) == mixrt.MIXRT_EINVAL
    assert lib.mixrt_raycast(R._h, None, 1, 8, 8, cams, buf.data_ptr(), None) == mixrt.MIXRT_EINVAL
    assert lib.mixrt_raycast(R._h, dm._h, 1, 8, 8, cams, buf.data_ptr() + 4, None) == mixrt.MIXRT_EINVAL
    assert lib.mixrt_raycast(R._h, dm._h, 1, 8, 8, cams, None, None) == mixrt.MIXRT_EINVAL
    assert lib.mixrt_raycast(R._h, dm._h, 1, 65536, 65536, cams, buf.data_ptr(),
                             None) == mixrt.MIXRT_EUNSUPPORTED
    cams[0].fov_y_deg = 0.0
    assert lib.mixrt_raycast(R._h, dm._h, 1, 8, 8, cams, buf.data_ptr(), None) == mixrt.MIXRT_EINVAL
    bad = mesh.faces.copy()
    bad[0, 0] = len(mesh.positions)
    with pytest.raises(mixrt.MixrtError):
        mixrt.DeviceMesh(R, synth.Mesh(positions=mesh.positions, faces=bad, uv=mesh.uv))
    dm.close()


# --------------------------------------------------------------------------
# The whole pipeline: ray cast, then render
# --------------------------------------------------------------------------

def _oracle_frame(sc, pix):
    """The oracle's own G-buffer at pix, then its render of those pixels.
    Returns (rgba [n, 4], ambiguous [n], hit [n])."""
    cfg = sc.cfg
    g0, _, _, amb = oracle.raycast_pixels(_cams(sc.cams), cfg.W, cfg.H, sc.mesh, pix,
                                          threads=oracle.max_threads())
    flat = sc.g0.reshape(-1, 4).copy()
    flat[pix] = g0.astype(np.float32)
    from dataclasses import replace
    sc2 = replace(sc, g0=flat.reshape(sc.g0.shape))
    rgba = oracle.OracleScene(sc2).render_pixels(pix, threads=oracle.max_threads())
    return rgba, amb, g0[:, 0] > 0


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("cfg", [synth.TINY64_MESH, synth.MESH720P], ids=lambda c: c.name)
def test_pipeline_parity(R, cfg, method):
    say("pipeline", cfg.name, method)
    sc = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    dm = mixrt.DeviceMesh(R, sc.mesh)
    gbuffer(R, method, dm, ds.cams, cfg.W, cfg.H, g1=False, out=(ds.g0, None))
    out = R.render(ds)
    R.sync()
    got = out.cpu().numpy()
    if cfg.rays <= 20000:
        pix = np.arange(cfg.rays)
    else:
        pix = np.unique(np.concatenate([np.random.default_rng(4).choice(cfg.rays, 400, replace=False),
                                        [0, cfg.rays - 1]]))
    ref, amb, hit = _oracle_frame(sc, pix)
    err = np.abs(got[pix][~amb] - ref[~amb]).max()
    say(f"  max |gpu - oracle| = {err:.3e} over {(~amb).sum()} px ({amb.sum()} ambiguous)")
    assert err <= FRAME_TOL
    assert np.all(np.isfinite(got))
    assert hit.mean() > 0.95                          # the room encloses the camera


def test_contexts_on_their_own_streams_agree_bitwise():
    """A context bound to a created (default-priority) stream gives the same
    rasterised G-buffer and frame as one on the current stream."""
    cfg = synth.TINY64_MESH
    sc = synth.make_scene(cfg)
    outs = []
    for stream in (None, torch.cuda.Stream()):
        r = mixrt.Renderer(0, stream=stream, sync_check=True)
        ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
        torch.cuda.synchronize()
        dm = mixrt.DeviceMesh(r, sc.mesh)
        r.rasterize(dm, ds.cams, cfg.W, cfg.H, g1=False, out=(ds.g0, None))
        out = r.render(ds)
        r.sync()
        outs.append((ds.g0.clone(), out.clone()))
        dm.close()
        r.close()
    assert torch.equal(outs[0][0], outs[1][0])
    assert torch.equal(outs[0][1], outs[1][1])


def test_frame_in_a_hip_graph_replays_like_eager():
    """rasterize + render captured in a HIP graph (no allocation, no memset
    in either): every replay, with eager work and synchronisation between
    replays, gives bitwise the eager G-buffer and frame."""
    cfg = synth.TINY64_MESH
    sc = synth.make_scene(cfg)
    s = torch.cuda.Stream()
    r = mixrt.Renderer(0, stream=s)        # no per-call synchronisation under capture
    ds = mixrt.DeviceScene.from_scene(sc, "cuda:0")
    dm = mixrt.DeviceMesh(r, sc.mesh)
    out = torch.empty((cfg.rays, 4), dtype=torch.float32, device="cuda:0")
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        r.rasterize(dm, ds.cams, cfg.W, cfg.H, g1=False, out=(ds.g0, None))
        r.render(ds, out)
    torch.cuda.synchronize()
    ref_g0, ref = ds.g0.clone(), out.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        r.rasterize(dm, ds.cams, cfg.W, cfg.H, g1=False, out=(ds.g0, None))
        r.render(ds, out)
    for _ in range(3):
        ds.g0.fill_(7.0)
        out.fill_(-1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(ds.g0, ref_g0)
        assert torch.equal(out, ref)
    dm.close()
    r.close()
