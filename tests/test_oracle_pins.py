"""Pins for the CPU oracle: each test checks an oracle function against
something other than itself -- exact quadrature, a library routine, exact
rational or integer arithmetic, or a closed form that the paper's equations or
the mathematics fix.  Each group names the passage it pins.
"""
from fractions import Fraction
from decimal import Decimal, getcontext

import numpy as np
import pytest
import scipy.special

import oracle
from paper_2312_11841_amd import synth

# --------------------------------------------------------------------------
# Stored values: fp16 upcast (tables, textures and weights are fp16)
# --------------------------------------------------------------------------


def test_half_to_double_matches_ieee_for_every_bit_pattern():
    bits = np.arange(65536, dtype=np.uint16)
    ours = oracle.half_to_double(bits)
    ref = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])


# --------------------------------------------------------------------------
# Level resolutions (geometric schedule from N_min to N_max)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("L,nmin,nmax", [(8, 16, 256), (16, 16, 4096), (16, 16, 8192),
                                         (4, 256, 4096), (1, 16, 16), (2, 16, 4096)])
def test_level_resolutions_closed_form(L, nmin, nmax):
    N = oracle.level_resolutions(L, nmin, nmax)
    assert N[0] == nmin and N[-1] == nmax
    assert np.all(np.diff(N) > 0) or L == 1
    if L > 1:
        getcontext().prec = 50
        b = (Decimal(nmax) / Decimal(nmin)) ** (Decimal(1) / Decimal(L - 1))
        for l in range(L):
            exact = Decimal(nmin) * b ** l
            # floor of the exact geometric value, except where that value is
            # an integer up to rounding (the guard in the schedule)
            assert abs(Decimal(int(N[l])) - exact) < 1
            assert Decimal(int(N[l])) <= exact + Decimal("1e-6")


def test_level_resolutions_power_of_two_endpoints_are_exact():
    # 16 * 2^(9 l / 15) hits 128 at l = 5 and 1024 at l = 10 for the 8192 grid
    N = oracle.level_resolutions(16, 16, 8192)
    assert N[5] == 128 and N[10] == 1024


# --------------------------------------------------------------------------
# Real spherical harmonics (Eq. 2's S and the view-direction encoding)
# --------------------------------------------------------------------------

def _product_quadrature():
    # Gauss-Legendre in cos(theta) x uniform in phi: exact for the products of
    # two harmonics of degree <= 3 (polynomials of degree <= 6).
    ct, wt = np.polynomial.legendre.leggauss(12)
    phis = np.arange(24) * (2 * np.pi / 24)
    pts, wts = [], []
    for c, w in zip(ct, wt):
        s = np.sqrt(1 - c * c)
        for p in phis:
            pts.append((s * np.cos(p), s * np.sin(p), c))
            wts.append(w * 2 * np.pi / 24)
    return np.array(pts), np.array(wts)


def test_sh_orthonormal_by_exact_quadrature():
    pts, wts = _product_quadrature()
    Y = oracle.sh_basis(16, pts)
    gram = (Y * wts[:, None]).T @ Y
    assert np.abs(gram - np.eye(16)).max() < 1e-12


def test_sh_matches_scipy_complex_harmonics():
    rng = np.random.default_rng(5)
    d = rng.normal(size=(64, 3))
    d /= np.linalg.norm(d, axis=1, keepdims=True)
    theta = np.arccos(np.clip(d[:, 2], -1, 1))
    phi = np.arctan2(d[:, 1], d[:, 0])
    Y = oracle.sh_basis(16, d)
    v = 0
    for l in range(4):
        for m in range(-l, l + 1):
            c = scipy.special.sph_harm_y(l, abs(m), theta, phi)  # has (-1)^m
            if m == 0:
                ref = c.real
            elif m > 0:
                ref = np.sqrt(2) * (-1) ** m * c.real
            else:
                ref = np.sqrt(2) * (-1) ** m * c.imag
            assert np.abs(Y[:, v] - ref).max() < 1e-12, (l, m)
            v += 1


def test_sh_constant_band_and_parity():
    d = np.array([0.3, -0.5, 0.812403840463596])
    assert oracle.sh_real(0, 0, d) == pytest.approx(0.5 / np.sqrt(np.pi), abs=1e-15)
    Y = oracle.sh_basis(16, d)
    Yn = oracle.sh_basis(16, -d)
    band = np.repeat(np.arange(4), [1, 3, 5, 7])
    assert np.allclose(Yn[0], Y[0] * (-1.0) ** band, atol=1e-14)
    # degree 1 along the axes: sqrt(3/(4 pi)) * (y, z, x)
    k1 = np.sqrt(3 / (4 * np.pi))
    assert np.allclose(oracle.sh_basis(4, [0, 0, 1])[0], [0.5 / np.sqrt(np.pi), 0, k1, 0],
                       atol=1e-14)
    assert np.allclose(oracle.sh_basis(4, [1, 0, 0])[0], [0.5 / np.sqrt(np.pi), 0, 0, k1],
                       atol=1e-14)
    assert np.allclose(oracle.sh_basis(4, [0, 1, 0])[0], [0.5 / np.sqrt(np.pi), k1, 0, 0],
                       atol=1e-14)


# --------------------------------------------------------------------------
# Camera rays (Sec. 3.1: a ray through each pixel)
# --------------------------------------------------------------------------

def _cam(R=np.eye(3), o=np.zeros(3), fov=60.0):
    c = np.zeros(16, np.float32)
    c[:12] = np.concatenate([R, np.asarray(o)[:, None]], 1).reshape(-1)
    c[12] = fov
    return c


def test_camera_rays_pinhole_geometry():
    W, H, fov = 64, 48, 60.0
    cam = _cam(fov=fov)
    # project every pixel centre on the plane z = -1
    proj = np.zeros((H, W, 2))
    for j in range(H):
        for i in range(W):
            o, d = oracle.camera_ray(cam, W, H, i, j)
            assert np.allclose(o, 0) and abs(np.linalg.norm(d) - 1) < 1e-14
            assert d[2] < 0
            proj[j, i] = d[:2] / -d[2]
    # equally spaced grid, square pixels, row 0 at the top (+y)
    sx = np.diff(proj[..., 0], axis=1)
    sy = np.diff(proj[..., 1], axis=0)
    assert np.allclose(sx, sx[0, 0], atol=1e-12) and np.allclose(sy, -sx[0, 0], atol=1e-12)
    # image centred on the optical axis; the top edge lies at tan(fov / 2)
    assert np.allclose(proj.mean(axis=(0, 1)), 0, atol=1e-12)
    top_edge = proj[0, 0, 1] + 0.5 * sx[0, 0]
    assert top_edge == pytest.approx(np.tan(np.deg2rad(fov / 2)), abs=1e-12)
    assert proj[0, 0, 1] > 0 and proj[0, 0, 0] < 0


def test_camera_pose_rotates_and_translates():
    a = np.deg2rad(30)
    R = np.array([[np.cos(a), 0, np.sin(a)], [0, 1, 0], [-np.sin(a), 0, np.cos(a)]])
    o0, d0 = oracle.camera_ray(_cam(), 16, 16, 3, 11)
    o1, d1 = oracle.camera_ray(_cam(R, [1.0, -2.0, 0.5]), 16, 16, 3, 11)
    Rf = R.astype(np.float32).astype(np.float64)
    assert np.allclose(o1, [1.0, -2.0, 0.5])
    assert np.allclose(d1, Rf @ d0 / np.linalg.norm(Rf @ d0), atol=1e-14)


# --------------------------------------------------------------------------
# Displacement texture fetch and Eq. 2 calibration
# --------------------------------------------------------------------------

def _bilinear_tex(R, coef, dtype=np.float32):
    jj, ii = np.mgrid[0:R, 0:R].astype(np.float64)
    a0, a1, a2, a3 = coef
    return (a0 + a1 * ii + a2 * jj + a3 * ii * jj)[..., None].astype(dtype)


def test_bilinear_reproduces_bilinear_functions_inside():
    R = 16
    coef = (0.25, 0.5, -0.75, 0.125)
    tex = _bilinear_tex(R, coef)
    rng = np.random.default_rng(1)
    for _ in range(200):
        u, v = rng.uniform(0.5 / R, 1 - 0.5 / R, 2)
        a, b = u * R - 0.5, v * R - 0.5   # texel-space coordinates, column from u
        ref = coef[0] + coef[1] * a + coef[2] * b + coef[3] * a * b
        assert oracle.tex_bilinear(tex, u, v)[0] == pytest.approx(ref, abs=1e-12)


def test_bilinear_texel_centres_and_clamp():
    R, V = 8, 3
    rng = np.random.default_rng(2)
    tex = rng.uniform(-1, 1, (R, R, V)).astype(np.float16)
    for j in range(R):
        for i in range(R):
            got = oracle.tex_bilinear(tex, (i + 0.5) / R, (j + 0.5) / R)
            assert np.array_equal(got, tex[j, i].astype(np.float64))
    # clamp to edge: outside the centre band only the edge texels count
    assert np.array_equal(oracle.tex_bilinear(tex, 0.0, 0.0), tex[0, 0].astype(np.float64))
    assert np.array_equal(oracle.tex_bilinear(tex, 1.0, 1.0), tex[-1, -1].astype(np.float64))
    got = oracle.tex_bilinear(tex, 0.0, (2 + 0.5) / R)
    assert np.array_equal(got, tex[2, 0].astype(np.float64))


def test_calibration_is_an_sh_weighted_length_along_the_ray():
    p = np.array([0.3, -1.0, 2.0])
    d = np.array([0.48, 0.6, -0.64])
    # zero map: the point does not move
    assert np.array_equal(oracle.calibrate(p, d, np.zeros(4)), p)
    # one-hot coefficient v moves the point by Y_v(d) along d
    pts, wts = _product_quadrature()
    Yall = oracle.sh_basis(8, d)[0]
    for v in range(8):
        m = np.zeros(8)
        m[v] = 0.5
        got = oracle.calibrate(p, d, m)
        assert np.allclose(got - p, 0.5 * Yall[v] * d, atol=1e-14)
    # constant-band coefficient: a view-independent offset 1/(2 sqrt(pi)) c
    got = oracle.calibrate(p, d, np.array([0.2]))
    assert np.allclose(got, p + 0.2 * 0.5 / np.sqrt(np.pi) * d, atol=1e-15)


# --------------------------------------------------------------------------
# Contraction (Sec. 2.1: Mip-NeRF 360 contraction into a ball of radius 2)
# --------------------------------------------------------------------------

def _uncube(x):
    return 4.0 * np.asarray(x) - 2.0


def test_contraction_identity_inside_unit_ball():
    rng = np.random.default_rng(3)
    for _ in range(100):
        q = rng.normal(size=3)
        q *= rng.uniform(0, 1) / np.linalg.norm(q)
        assert np.allclose(_uncube(oracle.contract(q)), q, atol=1e-14)


def test_contraction_closed_values_and_limits():
    assert np.allclose(oracle.contract([3.0, 0, 0]), [11 / 12, 0.5, 0.5], atol=1e-15)
    assert np.allclose(oracle.contract([0, -2.0, 0]), [0.5, (2 - 1.5) / 4, 0.5], atol=1e-15)
    u = np.array([2.0, -1.0, 2.0]) / 3.0
    far = _uncube(oracle.contract(1e9 * u))
    assert np.allclose(far, 2 * u, atol=1e-8)
    # continuity across the unit sphere and radial monotonicity
    inside = _uncube(oracle.contract((1 - 1e-9) * u))
    outside = _uncube(oracle.contract((1 + 1e-9) * u))
    assert np.allclose(inside, outside, atol=1e-8)
    radii = np.linspace(0.1, 50, 200)
    norms = [np.linalg.norm(_uncube(oracle.contract(r * u))) for r in radii]
    assert np.all(np.diff(norms) > 0) and max(norms) < 2


def test_cube_clamp():
    x = oracle.contract([1e300, 0, 0])
    assert np.all((x >= 0) & (x <= 1))


# --------------------------------------------------------------------------
# Hash encoding (Sec. 3.1: 8 nearest vertices, 1D table, trilinear)
# --------------------------------------------------------------------------

def _exact_corner(x32, N):
    """floor of the fp32 product x*N (IEEE multiply by numpy), via rationals."""
    pos = np.float32(x32) * np.float32(N)
    c = int(Fraction(float(pos)).__floor__())
    return min(max(c, 0), N - 1), Fraction(float(pos))


def _adversarial_positions(N):
    xs = [0.0, 1.0, np.nextafter(np.float32(1.0), np.float32(0.0))]
    for k in range(0, N + 1, max(1, N // 7)):
        x = np.float32(k) / np.float32(N)
        xs += [x, np.nextafter(x, np.float32(0)), np.nextafter(x, np.float32(2))]
    return np.array(xs, np.float32)


@pytest.mark.parametrize("cfg", [synth.TINY64, synth.VIEW720P])
def test_corners_match_exact_floor(cfg):
    N = oracle.level_resolutions(cfg.L, cfg.N_min, cfg.N_max)
    rng = np.random.default_rng(4)
    x = rng.uniform(0, 1, (3000, 3)).astype(np.float32)
    adv = []
    for l in range(cfg.L):
        a = _adversarial_positions(int(N[l]))
        adv.append(np.stack([a, a[::-1], np.roll(a, 3)], 1))
    x = np.concatenate([x] + adv)
    table = np.zeros((cfg.L, 1 << 10, cfg.F), np.float32)  # values unused here
    corner, idx, w, feat = oracle.hash_encode(x, table, cfg.N_min, cfg.N_max)
    for s in range(x.shape[0]):
        for l in range(cfg.L):
            for a in range(3):
                c, _ = _exact_corner(x[s, a], int(N[l]))
                assert corner[s, l, a] == c


def _dense_positions(N):
    """One query per cell, at the cell centre, so corner 0 is vertex v."""
    g = np.arange(N)
    v = np.stack(np.meshgrid(g, g, g, indexing="ij"), -1).reshape(-1, 3)
    return v, ((v + 0.5) / N).astype(np.float32)


@pytest.mark.parametrize("L, T, n_min, n_max, levels", [
    (synth.TINY64.L, synth.TINY64.T, synth.TINY64.N_min, synth.TINY64.N_max, (0, 1)),
    (2, 4096, 15, 31, (0,)),          # (N+1)^3 == T exactly: still one entry per vertex
])
def test_dense_levels_index_every_vertex_once(L, T, n_min, n_max, levels):
    N = oracle.level_resolutions(L, n_min, n_max)
    for l in levels:
        n = int(N[l])
        assert (n + 1) ** 3 <= T
        v, x = _dense_positions(n)
        table = np.zeros((L, T, 2), np.float32)
        corner, idx, _, _ = oracle.hash_encode(x, table, n_min, n_max)
        assert np.array_equal(corner[:, l], v)
        seen = {}
        for s in range(v.shape[0]):
            for beta in range(8):
                b = np.array([beta & 1, (beta >> 1) & 1, (beta >> 2) & 1])
                key = tuple(v[s] + b)
                i = int(idx[s, l, beta])
                assert seen.setdefault(key, i) == i
        assert sorted(seen.values()) == list(range((n + 1) ** 3))
        # x varies fastest: neighbours along x are adjacent entries
        assert seen[(1, 0, 0)] - seen[(0, 0, 0)] == 1


def test_hashed_indices_brute_force_and_structure():
    cfg = synth.VIEW720P
    N = oracle.level_resolutions(cfg.L, cfg.N_min, cfg.N_max)
    T = cfg.T
    rng = np.random.default_rng(6)
    x = rng.uniform(0, 1, (2000, 3)).astype(np.float32)
    table = np.zeros((cfg.L, 1 << 4, cfg.F), np.float32)
    # indices do not depend on the table values; use the real T via log2T
    corner, idx, _, _ = oracle.hash_encode(
        x, np.zeros((cfg.L, T, 1), np.float32), cfg.N_min, cfg.N_max)
    primes = (1, 2654435761, 805459861)
    for l in range(cfg.L):
        n = int(N[l])
        dense = (n + 1) ** 3 <= T
        for s in range(0, x.shape[0], 7):
            for beta in range(8):
                v = [int(corner[s, l, a]) + ((beta >> a) & 1) for a in range(3)]
                if dense:
                    ref = v[0] + v[1] * (n + 1) + v[2] * (n + 1) ** 2
                else:
                    h = 0
                    for a in range(3):
                        h ^= (v[a] * primes[a]) % (1 << 32)   # exact big-int product
                    ref = h % T
                assert int(idx[s, l, beta]) == ref
            if not dense:
                # x carries prime 1: along x an even vertex pairs with idx ^ 1
                if corner[s, l, 0] % 2 == 0:
                    assert idx[s, l, 1] == idx[s, l, 0] ^ 1
    del table


def test_trilinear_weights_partition_unity_and_vertices():
    cfg = synth.TINY64
    rng = np.random.default_rng(7)
    x = rng.uniform(0, 1, (500, 3)).astype(np.float32)
    table = np.zeros((cfg.L, cfg.T, cfg.F), np.float32)
    _, _, w, _ = oracle.hash_encode(x, table, cfg.N_min, cfg.N_max)
    assert np.all(w >= 0)
    assert np.abs(w.sum(-1) - 1).max() < 1e-12
    # exactly on a vertex: all weight on one corner (corner 0 inside, the far
    # corner at x = 1 where the cell is clamped)
    N = oracle.level_resolutions(cfg.L, cfg.N_min, cfg.N_max)
    for l in range(cfg.L):
        n = int(N[l])
        # vertex coordinates k / n whose fp32 product with n is exactly k
        ks = [k for k in range(1, n) if np.float32(np.float32(k / n) * np.float32(n)) == k]
        assert len(ks) >= 3
        xv = np.array([[ks[0] / n, ks[len(ks) // 2] / n, 0.0], [1.0, 1.0, 1.0]], np.float32)
        _, _, wv, _ = oracle.hash_encode(xv, table, cfg.N_min, cfg.N_max)
        assert wv[0, l, 0] == 1.0 and wv[1, l, 7] == 1.0


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_dense_interpolation_reproduces_affine_fields(dtype):
    cfg = synth.TINY64
    N = oracle.level_resolutions(cfg.L, cfg.N_min, cfg.N_max)
    table = np.zeros((cfg.L, cfg.T, cfg.F), dtype)
    A = np.array([[1.0, 3.0, -2.0, 5.0], [-4.0, 0.5, 2.0, -1.0]])  # per feature a.v + b
    for l in (0, 1):
        n = int(N[l])
        g = np.arange(n + 1)
        v = np.stack(np.meshgrid(g, g, g, indexing="ij"), -1).reshape(-1, 3)
        lin = v[:, 0] + v[:, 1] * (n + 1) + v[:, 2] * (n + 1) ** 2   # checked above
        for f in range(cfg.F):
            table[l, lin, f] = (v @ A[f, :3] + A[f, 3]).astype(dtype)
    rng = np.random.default_rng(8)
    x = rng.uniform(0, 1, (400, 3)).astype(np.float32)
    x[:5] = [[0, 0, 0], [1, 1, 1], [1, 0, 0.5], [0.25, 1, 0], [0.5, 0.5, 0.5]]
    _, _, _, feat = oracle.hash_encode(x, table, cfg.N_min, cfg.N_max)
    for l in (0, 1):
        n = int(N[l])
        pos = (x * np.float32(n)).astype(np.float64)   # the fp32 product, exactly
        for f in range(cfg.F):
            ref = pos @ A[f, :3] + A[f, 3]
            assert np.abs(feat[:, l * cfg.F + f] - ref).max() < 1e-9


# --------------------------------------------------------------------------
# MLP (Sec. 3.1: a small MLP turns the embedding into density and colour)
# --------------------------------------------------------------------------

def test_mlp_matches_numpy_matmul_chain():
    rng = np.random.default_rng(9)
    widths = (48, 64, 64, 4)
    ws = [rng.normal(0, 0.2, (widths[m], widths[m + 1])).astype(np.float16)
          for m in range(3)]
    x = rng.normal(0, 1, (300, 48))
    out = oracle.mlp(x, ws)
    h = x
    for m, w in enumerate(ws):
        h = h @ w.astype(np.float64)
        if m < 2:
            h = np.maximum(h, 0)
    assert np.allclose(out[:, 0], np.exp(h[:, 0]), rtol=1e-12)
    assert np.allclose(out[:, 1:], scipy.special.expit(h[:, 1:]), rtol=1e-12)


def test_mlp_removed_sums_inputs_per_component():
    x = np.arange(24, dtype=np.float64).reshape(2, 12) / 10.0
    out = oracle.mlp(x, [])
    o = x.reshape(2, 3, 4).sum(1)
    assert np.allclose(out[:, 0], np.exp(o[:, 0])) and np.allclose(out[:, 1:], scipy.special.expit(o[:, 1:]))


def test_mlp_identity_passes_input_through():
    x = np.array([[0.5, -0.25, 1.5, -3.0]] * 2 + [[2.0, 1.0, -1.0, 0.0]])
    eye = np.eye(4, dtype=np.float16)
    out = oracle.mlp(x, [eye, eye])
    relu = np.maximum(x, 0)
    assert np.allclose(out[:, 0], np.exp(relu[:, 0]))
    assert np.allclose(out[:, 1:], 1 / (1 + np.exp(-relu[:, 1:])))


# --------------------------------------------------------------------------
# Compositing (Eq. 1, with exclusive transmittance)
# --------------------------------------------------------------------------

def test_single_opaque_sample_returns_its_colour():
    s = np.array([[[1e9, 0.2, 0.7, 0.9]]])
    out = oracle.composite(s, 0.01, [0.5, 0.5, 0.5])
    assert np.allclose(out[0], [0.2, 0.7, 0.9, 1.0], atol=1e-15)
    # the same behind transparent samples
    s = np.array([[[0, 1, 1, 1], [0, 0, 0, 0], [1e9, 0.2, 0.7, 0.9], [5, 1, 0, 1]]], float)
    out = oracle.composite(s, 0.01, [0.5, 0.5, 0.5])
    assert np.allclose(out[0], [0.2, 0.7, 0.9, 1.0], atol=1e-15)


def test_zero_density_returns_background():
    rng = np.random.default_rng(10)
    s = rng.uniform(0, 1, (5, 8, 4))
    s[..., 0] = 0
    bg = rng.uniform(0, 1, (5, 3))
    out = oracle.composite(s, 0.3, bg)
    assert np.allclose(out[:, :3], bg, atol=1e-15) and np.all(out[:, 3] == 0)


def test_zero_length_interval_absorbs_nothing():
    """Eq. 1 with delta = 0: every alpha is 1 - exp(0) = 0, so the pixel is the
    background with alpha 0, also for a density that overflowed to infinity
    (whose product with 0 is otherwise undefined)."""
    rng = np.random.default_rng(12)
    s = rng.uniform(0, 1, (6, 5, 4))
    s[..., 0] = rng.exponential(3.0, (6, 5))
    s[0, :, 0] = np.inf
    s[1, 2, 0] = np.inf
    bg = rng.uniform(0, 1, (6, 3))
    out = oracle.composite(s, 0.0, bg)
    assert np.all(np.isfinite(out))
    assert np.array_equal(out[:, :3], bg) and np.all(out[:, 3] == 0)
    # and with delta > 0 an infinite density is one opaque sample
    out = oracle.composite(s[:1], 0.1, bg[:1])
    assert np.allclose(out[0], list(s[0, 0, 1:]) + [1.0], atol=0)


def test_compositing_weights_telescope_and_two_sample_form():
    rng = np.random.default_rng(11)
    K = 8
    s = rng.uniform(0, 3, (50, K, 4))
    s[..., 1:] = 1.0
    out = oracle.composite(s, 0.25, np.ones(3))
    assert np.abs(out[:, :3] - 1).max() < 1e-14   # sum_k T_k a_k + T_end = 1
    # two samples, running-product form
    s2, d = np.array([[[2.0, 0.1, 0.2, 0.3], [0.5, 0.9, 0.8, 0.7]]]), 0.4
    a1, a2 = 1 - np.exp(-2.0 * d), 1 - np.exp(-0.5 * d)
    bg = np.array([0.3, 0.6, 0.9])
    ref = a1 * s2[0, 0, 1:] + (1 - a1) * a2 * s2[0, 1, 1:] + (1 - a1) * (1 - a2) * bg
    out = oracle.composite(s2, d, bg)
    assert np.allclose(out[0, :3], ref, atol=1e-15)
    assert out[0, 3] == pytest.approx(1 - (1 - a1) * (1 - a2), abs=1e-15)


# --------------------------------------------------------------------------
# Steps 1-4 together: samples centred on the calibrated point, spaced delta
# --------------------------------------------------------------------------

def _small_scene(V=1, tex_val=0.0, K=5, delta=0.01, t=0.5):
    cfg = synth.TINY64.replace(name="pin", H=8, W=8, K=K, delta=delta, tex_R=4,
                               tex_V=V, L=2, log2_T=12, widths=(4, 16, 4))
    sc = synth.make_scene(cfg)
    sc.g0[..., 0] = t
    sc.tex[...] = 0
    sc.tex[..., 0] = tex_val
    return sc


@pytest.mark.parametrize("tex_val", [0.0, 0.3])
def test_samples_are_centred_on_calibrated_point(tex_val):
    sc = _small_scene(tex_val=tex_val)
    orc = oracle.OracleScene(sc)
    pix = np.arange(sc.cfg.rays)
    _, xd, hit = orc.pixel_samples(pix)
    assert np.all(hit == 1)
    s = 0.5 / np.sqrt(np.pi) * tex_val         # Y_00 times the constant channel
    for q in range(pix.size):
        j, i = divmod(q, sc.cfg.W)
        o, d = oracle.camera_ray(sc.cams[0], sc.cfg.W, sc.cfg.H, i, j)
        qk = _uncube(xd[q])                     # inside the unit ball: identity
        assert np.allclose(qk.mean(0), o + (0.5 + s) * d, atol=1e-12)
        steps = np.diff(qk, axis=0)
        assert np.allclose(steps, sc.cfg.delta * d, atol=1e-12)


def test_view_direction_sh_feeds_the_mlp():
    # zero table: the MLP sees only the 16 SH values of the ray direction, so
    # all K samples share (sigma, rgb) and compositing has a closed form
    cfg = synth.TINY64.replace(name="shpin", H=6, W=10, K=4, delta=0.05, L=2, log2_T=12,
                               view_sh_dim=16, widths=(2 * 2 + 16, 4))
    sc = synth.make_scene(cfg)
    sc.g0[..., 0] = 0.5
    sc.table[...] = 0
    Wt = sc.weights[0].astype(np.float64)
    assert Wt.shape == (20, 4)
    out = oracle.OracleScene(sc).render_pixels(np.arange(cfg.rays))
    assert 0.01 < out[:, 3].min() and out[:, 3].max() < 0.99      # neither clear nor opaque
    bg = np.array(sc.cams[0, 13:16], np.float64)
    for q in range(cfg.rays):
        j, i = divmod(q, cfg.W)
        _, d = oracle.camera_ray(sc.cams[0], cfg.W, cfg.H, i, j)
        o = oracle.sh_basis(16, d)[0] @ Wt[4:]
        T_end = np.exp(-cfg.K * np.exp(o[0]) * cfg.delta)
        rgb = scipy.special.expit(o[1:])
        assert np.allclose(out[q, :3], rgb * (1 - T_end) + bg * T_end, atol=1e-12)
        assert out[q, 3] == pytest.approx(1 - T_end, abs=1e-12)


def test_miss_pixels_return_background():
    sc = synth.make_scene(synth.TINY64_DENSE)
    sc.g0[0, 0, :4, 0] = [0.0, -1.0, np.nan, np.inf]
    out = oracle.OracleScene(sc).render_pixels(np.arange(5))
    bg = np.array(sc.cfg.bg)
    assert np.allclose(out[:4, :3], bg) and np.all(out[:4, 3] == 0)
    assert out[4, 3] > 0


def test_constant_field_reduces_to_one_mlp_query():
    # A constant table makes every feature the constant (weights sum to 1);
    # with K = 1 and a huge density the pixel is that query's colour: the
    # paper's one-query-per-pixel pipeline.
    cfg = synth.TINY64.replace(name="const", K=1, delta=1.0)
    sc = synth.make_scene(cfg)
    sc.table[...] = 0.375
    sc.weights[0] = np.full(sc.weights[0].shape, 0.1, np.float16)
    w_last = sc.weights[-1].astype(np.float32)
    w_last[:, 0] = 5.0
    sc.weights[-1] = w_last.astype(np.float16)
    hid = np.full(cfg.widths[1], 0.375 * cfg.widths[0] * float(np.float16(0.1)))
    o = hid @ sc.weights[-1].astype(np.float64)
    assert o[0] > 90                                   # opaque: alpha = 1
    out = oracle.OracleScene(sc).render_pixels(np.arange(0, cfg.rays, 97))
    assert np.allclose(out[:, :3], scipy.special.expit(o[1:]), atol=1e-12)
    assert np.allclose(out[:, 3], 1.0)


# --------------------------------------------------------------------------
# Eq. 2 as printed (SH vector x scale map), 8-bit maps, no displacement
# --------------------------------------------------------------------------

def test_u8_map_is_dequantised_affinely():
    R = 8
    jj, ii = np.mgrid[0:R, 0:R]
    q = (3 + 2 * ii + 5 * jj + ii * jj).astype(np.uint8)[..., None]   # bilinear in (i, j)
    qs, qo = 0.01, -0.7
    rng = np.random.default_rng(20)
    for _ in range(50):
        u, v = rng.uniform(0.5 / R, 1 - 0.5 / R, 2)
        a, b = u * R - 0.5, v * R - 0.5
        ref = qo + qs * (3 + 2 * a + 5 * b + a * b)
        assert oracle.map_bilinear(q, 1, u, v, qs, qo)[0] == pytest.approx(ref, abs=1e-12)
    # texel centre: exactly q_offset + q_scale * q
    assert oracle.map_bilinear(q, 1, 2.5 / R, 5.5 / R, qs, qo)[0] == pytest.approx(
        qo + qs * float(q[5, 2, 0]), abs=1e-15)


@pytest.mark.parametrize("disp", ["ray", "vec3"])
def test_u8_maps_use_their_own_affine_pairs_end_to_end(disp):
    # 8-bit coefficient and scale maps, each constant, with distinct affine
    # pairs: the mean sample must move by the dequantised values, so taking a
    # map's pair from the other map shows up as a wrong offset.
    cfg = synth.TINY64.replace(name="u8pin", H=8, W=8, K=3, delta=0.01, tex_R=4,
                               tex_dtype="u8", disp=disp, sh_degree=1, L=2, log2_T=12,
                               widths=(4, 16, 4))
    sc = synth.make_scene(cfg)
    sc.g0[..., 0] = 0.5
    sc.q_scale, sc.q_offset = (0.002, 0.004), (-0.25, 0.1)
    sc.tex[...] = 125                          # dequantises to exactly 0
    y00 = 0.5 / np.sqrt(np.pi)
    if disp == "ray":
        sc.tex[..., 0] = 200                   # m_0 = -0.25 + 0.002 * 200 = 0.15
        along, off = y00 * 0.15, np.zeros(3)
    else:
        nb = 4
        sc.tex[..., 0], sc.tex[..., nb], sc.tex[..., 2 * nb] = 225, 50, 175
        coef = -0.25 + 0.002 * np.array([225.0, 50.0, 175.0])    # (0.2, -0.15, 0.1)
        sc.scale[...] = 100                    # m_s = 0.1 + 0.004 * 100 = 0.5
        along, off = 0.0, 0.5 * y00 * coef
    _, xd, hit = oracle.OracleScene(sc).pixel_samples(np.arange(cfg.rays))
    assert np.all(hit == 1)
    for q in range(cfg.rays):
        j, i = divmod(q, cfg.W)
        o, d = oracle.camera_ray(sc.cams[0], cfg.W, cfg.H, i, j)
        assert np.allclose(_uncube(xd[q]).mean(0), o + (0.5 + along) * d + off, atol=1e-7)


def test_padding_channels_are_ignored():
    rng = np.random.default_rng(21)
    used = rng.uniform(-1, 1, (6, 6, 12)).astype(np.float32)
    padded = np.concatenate([used, rng.uniform(-9, 9, (6, 6, 4)).astype(np.float32)], -1)
    for _ in range(20):
        u, v = rng.uniform(-0.1, 1.1, 2)
        assert np.array_equal(oracle.map_bilinear(used, 12, u, v),
                              oracle.map_bilinear(padded, 12, u, v))


def test_vector_calibration_axis_by_axis():
    p = np.array([0.5, -0.25, 1.0])
    d = np.array([0.6, 0.0, -0.8])
    for D in range(4):
        nb = (D + 1) ** 2
        Y = oracle.sh_basis(nb, d)[0]
        assert np.array_equal(oracle.calibrate_vec3(p, d, np.zeros(3 * nb), nb, 0.7), p)
        for a in range(3):
            for v in range(nb):
                m = np.zeros(3 * nb)
                m[a * nb + v] = 0.4
                step = np.zeros(3)
                step[a] = 0.7 * 0.4 * Y[v]
                assert np.allclose(oracle.calibrate_vec3(p, d, m, nb, 0.7) - p, step, atol=1e-15)
        # the scale map scales the whole vector
        m = np.random.default_rng(D).uniform(-1, 1, 3 * nb)
        a1 = oracle.calibrate_vec3(p, d, m, nb, 1.0) - p
        assert np.allclose(oracle.calibrate_vec3(p, d, m, nb, 0.25) - p, 0.25 * a1, atol=1e-15)
        # constant band only: a view-independent offset Y_00 * m_s * c
        m = np.zeros(3 * nb)
        m[[0, nb, 2 * nb]] = [0.3, -0.2, 0.1]
        off = oracle.calibrate_vec3(p, d, m, nb, 0.5) - p
        assert np.allclose(off, 0.5 * 0.5 / np.sqrt(np.pi) * np.array([0.3, -0.2, 0.1]),
                           atol=1e-15)


def test_displacement_forms_agree_when_the_maps_vanish():
    base = synth.TINY64_DENSE.replace(H=16, W=16)
    pix = np.arange(256)
    zero_ray = synth.make_scene(base)
    zero_ray.tex[...] = 0
    ref = oracle.OracleScene(zero_ray).render_pixels(pix)
    none = synth.make_scene(base.replace(disp="none"))
    assert np.array_equal(oracle.OracleScene(none).render_pixels(pix), ref)
    vec = synth.make_scene(base.replace(disp="vec3", sh_degree=2))
    vec.g0, vec.table, vec.weights = zero_ray.g0, zero_ray.table, zero_ray.weights
    vec.scale[...] = 0                      # zero scale: no displacement
    assert np.array_equal(oracle.OracleScene(vec).render_pixels(pix), ref)


def test_samples_follow_the_vector_displacement():
    # inside the unit ball the cube map is affine, so the mean sample is
    # o + t d + m_s * S(m_SH, d): check it on a constant-band map
    cfg = synth.TINY64.replace(name="vecpin", H=8, W=8, K=3, delta=0.01, tex_R=4,
                               disp="vec3", sh_degree=1, L=2, log2_T=12, widths=(4, 16, 4))
    sc = synth.make_scene(cfg)
    sc.g0[..., 0] = 0.5
    sc.tex[...] = 0
    nb = 4
    sc.tex[..., 0], sc.tex[..., nb], sc.tex[..., 2 * nb] = 0.2, -0.1, 0.3
    sc.scale[...] = 0.5
    _, xd, _ = oracle.OracleScene(sc).pixel_samples(np.arange(cfg.rays))
    off = 0.5 * 0.5 / np.sqrt(np.pi) * np.array([0.2, -0.1, 0.3])
    for q in range(cfg.rays):
        j, i = divmod(q, cfg.W)
        o, d = oracle.camera_ray(sc.cams[0], cfg.W, cfg.H, i, j)
        assert np.allclose(_uncube(xd[q]).mean(0), o + 0.5 * d + off, atol=1e-7)
