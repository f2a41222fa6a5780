"""The pins must reject plausible mistakes: each case plants one mistake in a
copy of the oracle's C source (on the CPU), builds it, and requires the pin
suite to fail against that build."""
import concurrent.futures
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "mixrt_oracle.c")

MUTATIONS = {
    "prime_swap": ("(uint32_t)v[1] * 2654435761u) ^ ((uint32_t)v[2] * 805459861u)",
                   "(uint32_t)v[1] * 805459861u) ^ ((uint32_t)v[2] * 2654435761u)"),
    "xor_to_plus": ("((uint32_t)v[0] * 1u) ^ ((uint32_t)v[1]", "((uint32_t)v[0] * 1u) + ((uint32_t)v[1]"),
    "dense_strides": ("side * (uint64_t)v[1] + side * side * (uint64_t)v[2]",
                      "side * (uint64_t)v[2] + side * side * (uint64_t)v[1]"),
    "uv_swap": ("double a = u * R - 0.5, b = v * R - 0.5;", "double a = v * R - 0.5, b = u * R - 0.5;"),
    "no_half_texel": ("double a = u * R - 0.5, b = v * R - 0.5;", "double a = u * R, b = v * R;"),
    "inclusive_T": ("double T = exp(-optical);\n            double tau",
                    "double T = exp(-optical - s[4 * k] * delta);\n            double tau"),
    "weight_flip": ("wt *= bit ? fr[a] : 1.0 - fr[a];", "wt *= bit ? 1.0 - fr[a] : fr[a];"),
    "sh_sign": ("return sqrt(2.0) * k * p * sin((double)am * phi);",
                "return -sqrt(2.0) * k * p * sin((double)am * phi);"),
    "contract_norm": ("(2.0 - 1.0 / r) * (q[a] / r)", "(2.0 - 1.0 / r) * q[a]"),
    "fov_full": ("tan(0.5 * (double)cam[12]", "tan((double)cam[12]"),
    "row_up": ("-((double)j + 0.5 - 0.5 * H) / f", "((double)j + 0.5 - 0.5 * H) / f"),
    "sample_offset": ("((double)k - 0.5 * (double)(sc->K - 1)) * sc->delta", "((double)k) * sc->delta"),
    "relu_on_head": ("b[o] = (m < n_layers - 1 && acc < 0.0) ? 0.0 : acc;", "b[o] = (acc < 0.0) ? 0.0 : acc;"),
    "no_level_guard": ("pow(b, (double)l) + 1e-6)", "pow(b, (double)l))"),
    "calibration_sign": ("p_cali[r] = p[r] + s * d[r];", "p_cali[r] = p[r] - s * d[r];"),
    "corner_clamp": ("c0[a] = c < 0 ? 0 : (c > N - 1 ? N - 1 : c);", "c0[a] = c < 0 ? 0 : (c > N ? N : c);"),
    "subnormal_exp": ("v = ldexp((double)mant, -24);", "v = ldexp((double)mant, -25);"),
    "vec3_axis_stride": ("s += y[v] * m[a * nb + v];", "s += y[v] * m[v * 3 + a];"),
    "u8_offset": ("return m->q_offset + m->q_scale * (double)((const uint8_t *)m->data)[i];",
                  "return m->q_scale * (double)((const uint8_t *)m->data)[i];"),
    "scale_map_takes_coef_pair": ("sc->scale, sc->q_scale[1], sc->q_offset[1]};",
                                  "sc->scale, sc->q_scale[0], sc->q_offset[0]};"),
    "coef_map_takes_scale_pair": ("sc->tex, sc->q_scale[0], sc->q_offset[0]};",
                                  "sc->tex, sc->q_scale[1], sc->q_offset[1]};"),
    "dense_boundary_hashed": ("if (side * side * side <= T)", "if (side * side * side < T)"),
    "view_sh_scaled": ("hk[L * F + e] = sh[e];", "hk[L * F + e] = sh[e] * 0.5;"),
    "stored_channels": ("s += w[y][x] * map_value(m, ((int64_t)jb[y] * R + ia[x]) * m->C + c);",
                        "s += w[y][x] * map_value(m, ((int64_t)jb[y] * R + ia[x]) * nch + c);"),
    "no_background": ("out[4 * r + ch] = c[ch] + Tend * bg[3 * r + ch];", "out[4 * r + ch] = c[ch];"),
    "tie_to_higher_index": ("b1 + b2 <= 1.0 && t < best) {", "b1 + b2 <= 1.0 && t <= best) {"),
    "hits_behind": ("if (t > t_min && b1 >= 0.0", "if (b1 >= 0.0"),
    "uv_corner_swap": ("+ bb1 * uv[2 * fc[1] + k] + bb2 * uv[2 * fc[2] + k]",
                       "+ bb2 * uv[2 * fc[1] + k] + bb1 * uv[2 * fc[2] + k]"),
    "normal_flip": ("double nn = sqrt(n[0] * n[0] + n[1] * n[1] + n[2] * n[2]);\n    for (int k = 0; k < 3; ++k)\n        normal[k] = nn > 0.0 ? n[k] / nn",
                    "double nn = sqrt(n[0] * n[0] + n[1] * n[1] + n[2] * n[2]);\n    for (int k = 0; k < 3; ++k)\n        normal[k] = nn > 0.0 ? -n[k] / nn"),
    "q_uses_e2": ("q[0] = s[1] * e1[2] - s[2] * e1[1];", "q[0] = s[1] * e2[2] - s[2] * e2[1];"),
    "no_grazing_slack": ("return fmax(1.0, 0.1 / fmax(fabs(cosine), 1e-12));", "return 1.0;"),
    "no_depth_slack": ("double reach = best_i >= 0 ? best * (1.0 + eps_t * g) : INFINITY;",
                       "double reach = best_i >= 0 ? best : INFINITY;"),
    "gbuffer_t_min": ("uv, 1e-4, &t, bary, uvo, n, &ambiguous);", "uv, 1e-2, &t, bary, uvo, n, &ambiguous);"),
    "cosine_sign": ("*cosine = -det / sqrt", "*cosine = det / sqrt"),
    "no_near_miss": ("fmin(fmin(b1, b2), 1.0 - b1 - b2) > -eps_b * g)", "fmin(fmin(b1, b2), 1.0 - b1 - b2) > 0.0)"),
    'fr_from_c': ('fr[a] = (double)pos[a] - (double)c0[a];',
        'fr[a] = (double)pos[a] - (double)c;'),
    'alpha_no_delta': ('double tau = delta > 0.0 ? s[4 * k] * delta : 0.0;',
        'double tau = delta > 0.0 ? s[4 * k] : 0.0;'),
    'zero_delta_not_special': ('double tau = delta > 0.0 ? s[4 * k] * delta : 0.0;',
        'double tau = s[4 * k] * delta;'),
    'sigma_relu': ('out4[4 * s + 0] = exp(o[0]);',
        'out4[4 * s + 0] = o[0] > 0.0 ? o[0] : 0.0;'),
    'sigmoid_sign': ('out4[4 * s + c] = 1.0 / (1.0 + exp(-o[c]));',
        'out4[4 * s + c] = 1.0 / (1.0 + exp(o[c]));'),
    'sigma_relu_nomlp': ('out4[4 * s + 0] = exp(a[0]);',
        'out4[4 * s + 0] = a[0] > 0.0 ? a[0] : 0.0;'),
    'cube_map': ('double u = (c + 2.0) / 4.0;',
        'double u = (c + 1.0) / 2.0;'),
    'b_over_L': ('/ (double)(L - 1));',
        '/ (double)L);'),
    'pix_transpose': ('int j = (int)(rem / sc->W), i = (int)(rem % sc->W);',
        'int i = (int)(rem / sc->W), j = (int)(rem % sc->W);'),
    'pos_double': ('pos[a] = x[a] * (float)N;',
        'pos[a] = (float)((double)x[a] * (double)N + 1e-7);'),
    'bg_index': ('bg[c] = cam[13 + c];',
        'bg[c] = cam[12 + c];'),
    'tend_incl': ('double Tend = exp(-optical);',
        'double Tend = exp(-optical) * 0.5;'),
    't_gate': ('if (!(t > 0.0 && isfinite(t)))',
        'if (!(t >= 0.0 && isfinite(t)))'),
    'vec3_scale_ignored': ('p_cali[a] = p[a] + s * ms;',
        'p_cali[a] = p[a] + s;'),
    'no_hidden_relu': ('b[o] = (m < n_layers - 1 && acc < 0.0) ? 0.0 : acc;',
        'b[o] = acc;'),
    'weight_transpose': ('acc += orc_half_to_double(wm[(int64_t)k * no + o]) * a[k];',
        'acc += orc_half_to_double(wm[(int64_t)o * ni + k]) * a[k];'),
    'cam_transpose': ('d[r] = (double)cam[4 * r + 0] * dc[0] + (double)cam[4 * r + 1] * dc[1] +\n               (double)cam[4 * r + 2] * dc[2];',
        'd[r] = (double)cam[r] * dc[0] + (double)cam[4 + r] * dc[1] +\n               (double)cam[8 + r] * dc[2];'),
    'fov_uses_W': ('double f = 0.5 * (double)H / tan',
        'double f = 0.5 * (double)W / tan'),
    'no_dir_normalise': ('double inv = 1.0 / sqrt(n2);',
        'double inv = 1.0;'),
    'legendre_rec': ('(double)(ll + m - 1) * pmm) / (double)(ll - m);',
        '(double)(ll + m) * pmm) / (double)(ll - m);'),
    'sh_order': ('for (int m = -l; m <= l && v < n; ++m)',
        'for (int m = l; m >= -l && v < n; --m)'),
    'sh_cs_phase': ('pmm *= (double)(2 * i - 1) * s;',
        'pmm *= -(double)(2 * i - 1) * s;'),
    'bilinear_clamp_wrap': ('int ia[2] = {clampi(i0, 0, R - 1), clampi(i0 + 1, 0, R - 1)};',
        'int ia[2] = {(i0 + R) % R, (i0 + 1) % R};'),
    'bilinear_w': ('{(1 - wa) * wb, wa * wb}};',
        '{wa * wb, (1 - wa) * wb}};'),
    'contract_r_lt': ('double c = r <= 1.0 ? q[a]',
        'double c = r < 0.5 ? q[a]'),
    'half_norm_bias': ('v = ldexp((double)(mant + 1024), expo - 25);',
        'v = ldexp((double)(mant + 1024), expo - 24);'),
    'nomlp_mod': ('o[i % 4] += in[s * widths[0] + i];',
        'o[(i / (widths[0] / 4)) % 4] += in[s * widths[0] + i];'),
    'composite_T_update': ('double T = exp(-optical);\n            double tau',
        'double T = exp(-0.5 * optical);\n            double tau'),
    'b2_margin_missing': ('*ambiguous = best_i >= 0 && fmin(fmin(bb1, bb2), 1.0 - bb1 - bb2) < eps_b * graze(bcos);',
        '*ambiguous = best_i >= 0 && fmin(bb1, 1.0 - bb1 - bb2) < eps_b * graze(bcos);'),
    'no_edge_flag': ('*ambiguous = best_i >= 0 && fmin(fmin(bb1, bb2), 1.0 - bb1 - bb2) < eps_b * graze(bcos);',
        '*ambiguous = 0;'),
    'reach_unbounded': ('double reach = best_i >= 0 ? best * (1.0 + eps_t * g) : INFINITY;',
        'double reach = INFINITY;'),
    'miss_flag_off': ('double reach = best_i >= 0 ? best * (1.0 + eps_t * g) : INFINITY;',
        'double reach = best_i >= 0 ? best * (1.0 + eps_t * g) : -1.0;'),
    'uv_b0_swapped': ('uv_out[k] = uv ? b0 * uv[2 * fc[0] + k]',
        'uv_out[k] = uv ? bb1 * uv[2 * fc[0] + k]'),
    'miss_t_zero': ('g0[4 * q + 0] = f < 0 ? -1.0 : t;',
        'g0[4 * q + 0] = f < 0 ? 0.0 : t;'),
    'b1_b2_swap': ('bary[0] = bb1;\n    bary[1] = bb2;',
        'bary[0] = bb2;\n    bary[1] = bb1;'),
    'edge_ge': ('b1 >= 0.0 && b2 >= 0.0 && b1 + b2 <= 1.0 && t < best',
        'b1 > 0.0 && b2 > 0.0 && b1 + b2 < 1.0 && t < best'),
}


def _pins_against(name, work):
    """Build the oracle with mistake `name` planted and run both pin suites
    against it; returns (exit status, tail of their output)."""
    a, b = MUTATIONS[name]
    src = open(SRC).read()
    if src.count(a) != 1:
        return None, f"mutation anchor for {name} not found once"
    mut = os.path.join(work, f"{name}.c")
    lib = os.path.join(work, f"lib{name}.so")
    with open(mut, "w") as f:
        f.write(src.replace(a, b))
    subprocess.run(["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-shared",
                    "-fPIC", mut, "-o", lib, "-lm"], check=True)
    env = dict(os.environ, MIXRT_ORACLE_LIB=lib, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_mesh_pins.py"),
                        "-x", "-q", "-p", "no:cacheprovider"], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    return r.returncode, r.stdout[-2000:]


@pytest.fixture(scope="module")
def outcomes(tmp_path_factory):
    """name -> (exit status, output).  In a single process every planted
    mistake is built and checked up front, several at a time; under
    pytest-xdist the workers already run in parallel, so each checks only the
    mistakes of the tests it is given."""
    work = str(tmp_path_factory.mktemp("mutants"))
    if os.environ.get("PYTEST_XDIST_WORKER"):
        return _Lazy(work)
    workers = max(1, min(8, os.cpu_count() or 1))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        names = sorted(MUTATIONS)
        return dict(zip(names, ex.map(lambda n: _pins_against(n, work), names)))


class _Lazy(dict):
    def __init__(self, work):
        super().__init__()
        self.work = work

    def __missing__(self, name):
        self[name] = _pins_against(name, self.work)
        return self[name]


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_reject_planted_mistake(name, outcomes):
    rc, out = outcomes[name]
    assert rc is not None, out
    assert rc != 0, f"pins did not catch {name}:\n{out}"
