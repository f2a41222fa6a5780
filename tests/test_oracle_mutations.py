"""The pins must reject plausible mistakes: each case plants one mistake in a
copy of the oracle's C source (on the CPU), builds it, and requires the pin
suite to fail against that build."""
import os
import subprocess
import sys
import tempfile

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
    "inclusive_T": ("double T = exp(-optical);\n            double alpha",
                    "double T = exp(-optical - s[4 * k] * delta);\n            double alpha"),
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
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_reject_planted_mistake(name, tmp_path):
    a, b = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(a) == 1, f"mutation anchor for {name} not found once"
    mut = tmp_path / "mut.c"
    mut.write_text(src.replace(a, b))
    lib = tmp_path / "liboracle_mut.so"
    subprocess.run(["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-shared",
                    "-fPIC", str(mut), "-o", str(lib), "-lm"], check=True)
    env = dict(os.environ, MIXRT_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_mesh_pins.py"),
                        "-x", "-q", "-p", "no:cacheprovider"], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"pins did not catch {name}:\n{r.stdout[-2000:]}"
