"""Pins of the oracle's coarse-mesh hit (Fig. 2, step 1: the ray-mesh
intersection that yields the hit point p and its texture coordinate p_t).

The oracle solves every ray against every triangle in fp64 (Moller-Trumbore).
These pins hold it to closed forms, to an independent plane-then-inside
formulation written here in numpy, and to the geometry of known meshes."""
import numpy as np
import pytest

import oracle as O
from paper_2312_11841_amd import synth

QUAD = np.array([[-1, -1, -2], [3, -1, -2], [-1, 3, -2]], np.float32)
TRI = np.array([[0, 1, 2]], np.int32)


def _unit(v):
    v = np.asarray(v, np.float64)
    return v / np.linalg.norm(v)


def test_single_triangle_closed_form():
    """Plane z = -2, right angle at (-1, -1): p = t d, b1 = (px + 1) / 4,
    b2 = (py + 1) / 4, t = 2 / |dz|."""
    rng = np.random.default_rng(0)
    uv = rng.uniform(0, 1, (3, 2)).astype(np.float32)
    for _ in range(50):
        a, b = rng.uniform(-0.45, 0.9, 2)
        if a + b > 0.9:
            continue
        d = _unit([a, b, -1.0])
        r = O.ray_mesh([0, 0, 0], d, QUAD, TRI, uv)
        assert r["tri"] == 0 and not r["ambiguous"]
        assert r["t"] == pytest.approx(2.0 / -d[2], rel=1e-14)
        b1, b2 = (2 * a + 1) / 4, (2 * b + 1) / 4
        np.testing.assert_allclose(r["bary"], [b1, b2], rtol=0, atol=1e-14)
        want = (1 - b1 - b2) * uv[0] + b1 * uv[1] + b2 * uv[2]
        np.testing.assert_allclose(r["uv"], want, rtol=0, atol=1e-14)
        np.testing.assert_allclose(r["normal"], [0, 0, 1], atol=1e-15)
        # the cosine between the ray and the unit face normal e1 x e2 = +z:
        # d_z, negative for a ray against the normal, positive once rewound
        t, c1, c2, cos = O.ray_triangle([0, 0, 0], d, QUAD, TRI, 0)
        assert (t, c1, c2) == pytest.approx((r["t"], b1, b2), abs=1e-14)
        assert cos == pytest.approx(d[2], abs=1e-15) and cos < 0
        assert O.ray_triangle([0, 0, 0], d, QUAD, TRI[:, [0, 2, 1]], 0)[3] == pytest.approx(
            -d[2], abs=1e-15)


def test_uv_reproduces_an_affine_map():
    """Vertex uv drawn from an affine map of position: the interpolated uv at
    the hit equals the map at the hit point, for any triangle."""
    rng = np.random.default_rng(1)
    A, c = rng.normal(size=(2, 3)), rng.normal(size=2)
    for _ in range(30):
        tri = rng.normal(size=(3, 3)).astype(np.float32) + np.array([0, 0, -5], np.float32)
        g = tri.astype(np.float64).mean(0) + 0.1 * rng.normal(size=3)
        o = rng.normal(size=3)
        d = _unit(g - o)
        uv = (tri.astype(np.float64) @ A.T + c).astype(np.float32)
        r = O.ray_mesh(o, d, tri, TRI, uv)
        if r["tri"] < 0:
            continue
        p = o + r["t"] * d
        np.testing.assert_allclose(r["uv"], A @ p + c, atol=2e-6)  # uv stored in f32


def test_misses():
    d = _unit([0.1, 0.1, -1.0])
    assert O.ray_mesh([0, 0, 0], -d, QUAD, TRI)["tri"] == -1            # behind the origin
    assert O.ray_mesh([0, 0, 0], [1, 0, 0], QUAD, TRI)["tri"] == -1     # parallel to the plane
    for out in ([-1.5, 0.5], [0.5, -1.5], [1.6, 1.6]):                  # beyond each edge
        r = O.ray_mesh([0, 0, 0], _unit([out[0] / 2, out[1] / 2, -1.0]), QUAD, TRI)
        assert r["tri"] == -1 and not r["ambiguous"]
    # the origin on the plane: t = 0 is not a hit (t must exceed t_min)
    assert O.ray_mesh([0, 0, -2], [0, 0, -1], QUAD, TRI)["tri"] == -1
    assert O.ray_mesh([0, 0, -2 + 5e-5], [0, 0, -1], QUAD, TRI)["tri"] == -1
    assert O.ray_mesh([0, 0, -2 + 5e-4], [0, 0, -1], QUAD, TRI)["tri"] == 0


def test_nearest_of_stacked_triangles_in_either_order():
    far = QUAD + np.array([0, 0, -1], np.float32)
    d = _unit([0.2, 0.1, -1.0])
    for pos, want in ((np.concatenate([QUAD, far]), 0), (np.concatenate([far, QUAD]), 1)):
        r = O.ray_mesh([0, 0, 0], d, pos, np.array([[0, 1, 2], [3, 4, 5]], np.int32))
        assert r["tri"] == want and not r["ambiguous"]
        assert r["t"] == pytest.approx(2.0 / -d[2], rel=1e-14)


def test_equal_distance_goes_to_the_lower_index_and_is_ambiguous():
    pos = np.concatenate([QUAD, QUAD[[1, 2, 0]], QUAD])
    faces = np.array([[0, 1, 2], [3, 4, 5], [6, 7, 8]], np.int32)
    r = O.ray_mesh([0, 0, 0], _unit([0.2, 0.1, -1.0]), pos, faces)
    assert r["tri"] == 0 and r["ambiguous"]
    r = O.ray_mesh([0, 0, 0], _unit([0.2, 0.1, -1.0]), pos, faces[::-1].copy())
    assert r["tri"] == 0 and r["ambiguous"]   # index 0 of the reversed list


def test_a_second_surface_just_behind_is_ambiguous():
    """A clear hit with a second, clearly hit triangle behind it: within the
    depth slack t (1 + 1e-4) the pixel is ambiguous, well beyond it is not."""
    d = _unit([0.2, 0.1, -1.0])
    faces = np.array([[0, 1, 2], [3, 4, 5]], np.int32)
    for gap, amb in ((3e-5, True), (1e-3, False)):
        behind = QUAD * np.array([1, 1, 1 + gap], np.float32)
        r = O.ray_mesh([0, 0, 0], d, np.concatenate([QUAD, behind]), faces)
        assert r["tri"] == 0 and r["ambiguous"] == amb
        assert r["t"] == pytest.approx(2.0 / -d[2], rel=1e-14)


def test_shared_edge_is_ambiguous_centre_is_not():
    pos = np.array([[-1, -1, -2], [1, -1, -2], [1, 1, -2], [-1, 1, -2]], np.float32)
    faces = np.array([[0, 1, 2], [0, 2, 3]], np.int32)
    r = O.ray_mesh([0, 0, 0], [0, 0, -1], pos, faces)        # on the diagonal
    assert r["tri"] in (0, 1) and r["ambiguous"]
    r = O.ray_mesh([0, 0, 0], _unit([0.25, -0.25, -1]), pos, faces)
    assert r["tri"] == 0 and not r["ambiguous"]
    r = O.ray_mesh([0, 0, 0], _unit([-0.25, 0.25, -1]), pos, faces)
    assert r["tri"] == 1 and not r["ambiguous"]
    # just outside the square: a near miss is ambiguous, a clear miss is not
    assert O.ray_mesh([0, 0, 0], _unit([0.5 + 2e-5, 0.1, -1]), pos, faces)["ambiguous"]
    assert not O.ray_mesh([0, 0, 0], _unit([0.6, 0.1, -1]), pos, faces)["ambiguous"]
    # a hit 1e-3 from the edge y = -1 (barycentric margin 5e-4): clear at
    # normal incidence, ambiguous for a ray that skims the plane at cos 0.02
    hit = np.array([0.0, -1.0 + 1e-3, -2.0])
    for d, amb in ((_unit([0, 0, -1]), False), (_unit([0.0, 1.0, -0.02]), True)):
        r = O.ray_mesh(hit - d, d, pos, faces)
        assert r["tri"] == 0 and r["ambiguous"] == amb


def _plane_inside_nearest(o, d, pos, faces, t_min=1e-4):
    """An independent formulation: intersect each triangle's plane, then keep
    hits whose three edge functions n . ((b - a) x (p - a)) agree in sign."""
    P = pos.astype(np.float64)[faces]                  # [nf, 3, 3]
    a, b, c = P[:, 0], P[:, 1], P[:, 2]
    n = np.cross(b - a, c - a)
    den = n @ d
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.einsum("ij,ij->i", n, a - o) / den
    p = o + t[:, None] * d
    e = [np.einsum("ij,ij->i", n, np.cross(y - x, p - x)) for x, y in ((a, b), (b, c), (c, a))]
    ok = (den != 0) & (t > t_min) & (e[0] >= 0) & (e[1] >= 0) & (e[2] >= 0)
    if not ok.any():
        return -1, np.inf
    t = np.where(ok, t, np.inf)
    i = int(np.argmin(t))
    return i, t[i]


def test_brute_force_agrees_with_an_independent_formulation():
    rng = np.random.default_rng(3)
    v, f = synth._icosphere(2)
    room = (v * (1.0 + 0.1 * rng.uniform(-1, 1, (len(v), 1)))) * 3.0
    blobs = [v * rng.uniform(0.2, 0.5) + rng.uniform(-1.5, 1.5, 3) for _ in range(4)]
    pos = np.concatenate([room] + blobs).astype(np.float32)
    faces = np.concatenate([f + k * len(v) for k in range(5)]).astype(np.int32)
    checked = 0
    for _ in range(300):
        o = rng.uniform(-0.3, 0.3, 3)
        d = _unit(rng.normal(size=3))
        r = O.ray_mesh(o, d, pos, faces)
        i, t = _plane_inside_nearest(o, d, pos, faces)
        if r["ambiguous"]:
            continue
        checked += 1
        assert r["tri"] == i
        assert r["t"] == pytest.approx(t, rel=1e-10)
        bt = O.ray_triangle(o, d, pos, faces, i)
        assert bt[0] == r["t"] and min(bt[1], bt[2], 1 - bt[1] - bt[2]) >= 0
    assert checked > 250


def test_icosphere_from_inside():
    """From the centre of a unit icosphere every ray hits, between the nearest
    face plane and the circumscribed sphere, on the face whose plane the ray
    meets, with a unit normal orthogonal to both edges."""
    v, f = synth._icosphere(3)
    pos, faces = v.astype(np.float32), f.astype(np.int32)
    P = pos.astype(np.float64)[faces]
    n = np.cross(P[:, 1] - P[:, 0], P[:, 2] - P[:, 0])
    inr = np.abs(np.einsum("ij,ij->i", n / np.linalg.norm(n, axis=1, keepdims=True), P[:, 0]))
    rng = np.random.default_rng(4)
    for _ in range(200):
        d = _unit(rng.normal(size=3))
        r = O.ray_mesh([0, 0, 0], d, pos, faces)
        assert r["tri"] >= 0
        assert inr.min() * (1 - 1e-12) <= r["t"] <= 1.0 + 1e-6
        e1 = P[r["tri"], 1] - P[r["tri"], 0]
        e2 = P[r["tri"], 2] - P[r["tri"], 0]
        assert abs(np.linalg.norm(r["normal"]) - 1) < 1e-14
        assert abs(r["normal"] @ e1) < 1e-12 and abs(r["normal"] @ e2) < 1e-12
        assert (r["normal"] @ np.cross(e1, e2)) > 0


def test_raycast_pixels_of_a_wall():
    """A camera looking down -z at a square wall z = -5: each pixel's t is
    5 / -d_z of its ray, uv is the wall's affine map, pixels past the wall miss."""
    W, H, fov = 24, 16, 60.0
    cam = np.zeros(16, np.float32)
    cam[:12] = np.concatenate([np.eye(3), np.zeros((3, 1))], 1).reshape(-1)
    cam[12] = fov
    half = 2.0
    pos = np.array([[-half, -half, -5], [half, -half, -5], [half, half, -5], [-half, half, -5]],
                   np.float32)
    faces = np.array([[0, 1, 2], [0, 2, 3]], np.int32)
    uv = (pos[:, :2] + half) / (2 * half)
    mesh = synth.Mesh(positions=pos, faces=faces, uv=uv.astype(np.float32))
    pix = np.arange(W * H)
    g0, nrm, tri, amb = O.raycast_pixels(cam[None], W, H, mesh, pix)
    f = 0.5 * H / np.tan(np.deg2rad(fov) / 2)
    j, i = np.divmod(pix, W)
    dc = np.stack([(i + 0.5 - W / 2) / f, -(j + 0.5 - H / 2) / f, -np.ones(W * H)], 1)
    d = dc / np.linalg.norm(dc, axis=1, keepdims=True)
    t = 5.0 / -d[:, 2]
    p = t[:, None] * d
    inside = (np.abs(p[:, 0]) < half) & (np.abs(p[:, 1]) < half)
    assert inside.any() and (~inside).any()
    ok = ~amb
    np.testing.assert_array_equal((tri >= 0)[ok], inside[ok])
    hit = ok & inside
    np.testing.assert_allclose(g0[hit, 0], t[hit], rtol=1e-13)
    np.testing.assert_allclose(g0[hit, 1:3], (p[hit, :2] + half) / (2 * half), atol=1e-7)
    np.testing.assert_allclose(nrm[hit], np.tile([0, 0, 1.0], (hit.sum(), 1)), atol=1e-15)
    assert np.all(g0[~inside & ok, 0] == -1.0)
    # the wall's lower-right triangle holds the pixels below its diagonal y = x
    np.testing.assert_array_equal(tri[hit] == 0, p[hit, 1] < p[hit, 0])


def test_raycast_pixels_without_uv_gives_zero_uv():
    """A mesh without texture coordinates: hits keep t and the normal, uv is 0."""
    W, H = 6, 5
    cam = np.zeros(16, np.float32)
    cam[:12] = np.concatenate([np.eye(3), np.zeros((3, 1))], 1).reshape(-1)
    cam[12] = 60.0
    pos = np.array([[-9, -9, -3], [9, -9, -3], [0, 9, -3]], np.float32)
    mesh = synth.Mesh(positions=pos, faces=TRI, uv=None)
    g0, nrm, tri, _ = O.raycast_pixels(cam[None], W, H, mesh, np.arange(W * H))
    assert np.all(tri == 0)
    assert np.all(g0[:, 1:] == 0)
    with_uv = synth.Mesh(positions=pos, faces=TRI, uv=np.ones((3, 2), np.float32))
    g0u, nrmu, _, _ = O.raycast_pixels(cam[None], W, H, with_uv, np.arange(W * H))
    np.testing.assert_array_equal(g0[:, 0], g0u[:, 0])
    np.testing.assert_array_equal(nrm, nrmu)
    np.testing.assert_allclose(g0u[:, 1:3], 1.0, atol=1e-12)


def test_raycast_pixels_minimum_hit_distance():
    """The G-buffer takes hits beyond t = 1e-4 only: a wall 2e-3 in front of
    the camera is hit by every pixel, one 5e-5 in front by none."""
    W, H = 8, 6
    cam = np.zeros(16, np.float32)
    cam[:12] = np.concatenate([np.eye(3), np.zeros((3, 1))], 1).reshape(-1)
    cam[12] = 60.0
    faces = np.array([[0, 1, 2], [0, 2, 3]], np.int32)
    for z, hit in ((2e-3, True), (5e-5, False)):
        pos = np.array([[-1, -1, -z], [1, -1, -z], [1, 1, -z], [-1, 1, -z]], np.float32)
        mesh = synth.Mesh(positions=pos, faces=faces, uv=np.zeros((4, 2), np.float32))
        g0, _, tri, _ = O.raycast_pixels(cam[None], W, H, mesh, np.arange(W * H))
        assert np.all((tri >= 0) == hit)
        if hit:
            assert np.all((g0[:, 0] >= np.float32(2e-3)) & (g0[:, 0] < 3e-3))


def test_procedural_mesh_is_closed_and_seeded():
    m = synth.make_mesh(5, room_level=3, n_objects=6, object_level=1, n_boxes=3, box_div=2)
    again = synth.make_mesh(5, room_level=3, n_objects=6, object_level=1, n_boxes=3, box_div=2)
    np.testing.assert_array_equal(m.positions, again.positions)
    np.testing.assert_array_equal(m.faces, again.faces)
    assert m.faces.min() == 0 and m.faces.max() == len(m.positions) - 1
    assert np.all((m.uv >= 0) & (m.uv <= 1))
    # every component is closed: each undirected edge bounds exactly two faces,
    # once in each direction (a consistently wound surface)
    e = np.concatenate([m.faces[:, [0, 1]], m.faces[:, [1, 2]], m.faces[:, [2, 0]]])
    P = m.positions
    key = np.round(np.concatenate([P[e[:, 0]], P[e[:, 1]]], 1), 5)
    fwd = {tuple(k) for k in key}
    rev = {tuple(np.concatenate([k[3:], k[:3]])) for k in key}
    assert fwd == rev and len(fwd) == len(key)
