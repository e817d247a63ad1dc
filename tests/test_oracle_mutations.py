"""The pins have teeth: plant plausible mistakes in a private copy of the oracle's
C source or of its Python driver (on the CPU only), rebuild or reload it, and
check that at least one pin fails for each planted mistake.  The real oracle is
never modified.
"""
import importlib.util
import os
import subprocess

import pytest

import test_oracle_pins as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "kmq_oracle.c")

MUTATIONS = {
    "sign1_wrong_sign_of_T": ("int32_t s = 2 * D - T;", "int32_t s = 2 * D + T;"),
    "bit_order_msb_first": ("(row[i >> 5] >> (i & 31))", "(row[i >> 5] >> (31 - (i & 31)))"),
    "f32_dropped_factor_2": ("double s = cn[j] - 2.0 * dot;", "double s = cn[j] - dot;"),
    "sq8_mean_floor": ("(2 * S[(int64_t)j * d + i] + cnt[j]) / (2 * cnt[j])", "S[(int64_t)j * d + i] / cnt[j]"),
    "split_sign_of_p": ("Z[(int64_t)j * d + i] = t * (even ? up : dn);", "Z[(int64_t)j * d + i] = t * (even ? dn : up);"),
    "sq8_truncating_round": ("float t = rintf((X[r * d + i] - lo[i]) * inv);",
                             "float t = floorf((X[r * d + i] - lo[i]) * inv);"),
    "alpha_inverted": ("(float)(s2 / s1)", "(float)(s1 / s2)"),
    "sign_bit_at_zero": ("if (ri > 0.0f)", "if (ri >= 0.0f)"),
    "project_transposed_W": ("(double)W[(int64_t)i * dout + o]", "(double)W[(int64_t)o * d + i]"),
    "ties_to_largest": ("if (j == 0 || s < bs) {\n        bs = s;\n        best = j;\n      }\n    }\n    a[r] = best;\n"
                        "    if (dist) {\n      double e",
                        "if (j == 0 || s <= bs) {\n        bs = s;\n        best = j;\n      }\n    }\n    a[r] = best;\n"
                        "    if (dist) {\n      double e"),
    "sign1_prep_no_centering": ("float t = fabsf(c[i] - m[i]);", "float t = fabsf(c[i]);"),
    "update_sign1_drops_minus": ("-(double)alpha[r]", "0.0"),
    "bf16_truncates": ("double q = rint(ldexp((double)x, -se));", "double q = trunc(ldexp((double)x, -se));"),
    "bf16_ties_away_from_zero": ("double q = rint(ldexp((double)x, -se));", "double q = round(ldexp((double)x, -se));"),
    "bf16_keeps_9_bits": ("int se = e - 8 < -133 ? -133 : e - 8;", "int se = e - 9 < -133 ? -133 : e - 9;"),
    "rabitq_bias_term_sign": ("b * (float)(2 * P - d)", "b * (float)(d - 2 * P)"),
    "rabitq_sq4_16_levels": ("(hi - lo) / 15.0f", "(hi - lo) / 16.0f"),
    "rabitq_drops_T": ("(float)(2 * D - T)", "(float)(2 * D)"),
    "lvq4_A_sign_of_bias": ("par[4 * r + 2] = fmaf(s, (float)S, db);", "par[4 * r + 2] = fmaf(s, (float)S, -db);"),
    "lvq4_drops_bx_sy_Sy": ("fmaf(bx * sy, (float)yS[j], fmaf(by, Ax, (sx * sy) * (float)dot))",
                            "fmaf(by, Ax, (sx * sy) * (float)dot)"),
    "lvq4_16_levels": ("const float s = hi > lo ? (hi - lo) / 15.0f : 1.0f;",
                       "const float s = hi > lo ? (hi - lo) / 16.0f : 1.0f;"),
    "prune_factor_not_squared": ("return g * g * (double)D / (double)d;", "return g * (double)D / (double)d;"),
    "prune_factor_inverted": ("return g * g * (double)D / (double)d;", "return g * g * (double)d / (double)D;"),
    "prune_test_not_strict": ("if (p > tau * orc_prune_factor(D, d, eps0)) {", "if (p >= tau * orc_prune_factor(D, d, eps0)) {"),
    "prune_sq8_test_not_strict": ("if ((float)p > lim) {", "if ((float)p >= lim) {"),
    "prune_previous_centroid_dropped": ("    int32_t best = pj;\n    double bd = tau;", "    int32_t best = pj;\n    double bd = 1e300;"),
    "prune_ties_to_larger": ("if (p < bd || (p == bd && j < best)) {", "if (p < bd || (p == bd && j > best)) {"),
    "prune_first_checkpoint_skipped": ("for (int32_t D = d_front; D < d; D += step) { /* checkpoints */",
                                       "for (int32_t D = d_front + step; D < d; D += step) { /* checkpoints */"),
    "hybrid_front_row_stride_d": ("(double)front[r * d0 + i]", "(double)front[r * d + i]"),
    "hybrid_front_adds_m": ("C[(int64_t)j * d + i] = i < d0 ? Z[(int64_t)j * d + i] : m[i] + Z[(int64_t)j * d + i];",
                            "C[(int64_t)j * d + i] = m[i] + Z[(int64_t)j * d + i];"),
}

# mistakes in the Python driver (hierarchical k-means, hybrid initialisation and update)
PY_MUTATIONS = {
    "fine_init_first_members": ("(np.arange(k_i, dtype=np.int64) * n_i) // k_i", "np.arange(k_i, dtype=np.int64)"),
    "fine_offsets_without_leading_zero": ("off = np.concatenate([[0], np.cumsum(k_i)])", "off = np.cumsum(k_i)"),
    "fine_remainder_ties_to_larger_index": ("key=lambda i: (-rems[i], i)", "key=lambda i: (-rems[i], -i)"),
    "fine_share_by_n_not_n_minus_1": ("w = v - 1 if v > 0 else 0", "w = v"),
    "refine_skipped": ("    if iters_refine > 0:\n        C, a, Jr", "    if iters_refine > 1:\n        C, a, Jr"),
    "meso_count_floor": ("return max(1, r + 1 if k - r * r > r else r)", "return max(1, r)"),
    "hybrid_init_front_not_copied": ('C[:, :d0] = P["front"][idx]', "C[:, :d0] = 0.0"),
    "hybrid_init_tail_without_m": ('C = sign1_decode(P["bits"][idx], P["alpha"][idx], P["d"], P["m"], d0)',
                                   'C = sign1_decode(P["bits"][idx], P["alpha"][idx], P["d"], np.zeros(P["d"], np.float32), d0)'),
    "hybrid_update_without_front": ('policy, front=P["front"], d0=P["d0"])', 'policy)'),
    "sqrt_rule_rounds_down": ("out.append(r + 1 if v - r * r > r else r)", "out.append(r)"),
    "sqrt_rule_rounds_half_down": ("out.append(r + 1 if v - r * r > r else r)",
                                   "out.append(r + 1 if v - r * r > r + 1 else r)"),
    "sqrt_rule_empty_gets_one": ("        if v <= 0:\n            out.append(0)", "        if v <= 0:\n            out.append(1)"),
}

PINS = [name for name in dir(pins) if name.startswith("test_")]
PY_SRC = os.path.join(ROOT, "oracle", "__init__.py")


def _load_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, name
    mutated = src.replace(old, new)
    cfile = tmp_path / f"{name}.c"
    cfile.write_text(mutated)
    hdr = os.path.join(ROOT, "oracle")
    so = tmp_path / f"{name}.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
                           "-I", hdr, "-o", str(so), str(cfile), "-lm"])
    spec = importlib.util.spec_from_file_location(f"oracle_mutant_{name}", os.path.join(ROOT, "oracle", "__init__.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod._LIB_PATH = str(so)
    mod._lib = None
    return mod


def _load_py_mutant(tmp_path, name, old, new):
    src = open(PY_SRC).read()
    assert src.count(old) == 1, name
    pyfile = tmp_path / f"{name}.py"
    pyfile.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location(f"oracle_py_mutant_{name}", str(pyfile))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod._LIB_PATH = os.path.join(ROOT, "oracle", "libkmq_oracle.so")
    mod._lib = None
    return mod


def _run_pin(fn, mod):
    import inspect
    params = inspect.signature(fn).parameters
    if "fmt" in params:
        for fmt in ("f32", "sq8"):
            fn(mod, fmt)
    else:
        fn(mod)


@pytest.mark.parametrize("name", sorted(MUTATIONS) + sorted(PY_MUTATIONS))
def test_planted_mistake_is_caught(tmp_path, name):
    if name in MUTATIONS:
        mod = _load_mutant(tmp_path, name, *MUTATIONS[name])
    else:
        mod = _load_py_mutant(tmp_path, name, *PY_MUTATIONS[name])
    failed = []
    for pin in PINS:
        try:
            _run_pin(getattr(pins, pin), mod)
        except Exception:  # noqa: BLE001 - any failure of a pin counts as caught
            failed.append(pin)
    assert failed, f"no pin caught the planted mistake {name}"
