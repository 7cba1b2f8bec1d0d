"""The pins are strong enough: every planted slip in the oracle is caught.

Each mutant is a copy of ``oracle/lamb_oracle.c`` with one textual edit (a
dropped term, a wrong sign, coefficient or exponent, swapped operands, a
missing clamp branch, ...). It is compiled into a temporary library and run
against every pin; at least one pin must fail. Mistakes are planted only in
this CPU-side copy, never in the shipped oracle or on a GPU.
"""

import os
import shutil

import pytest

import oracle
import oracle_pins

# (name, original text, replacement, which occurrence: 0 = first, 1 = second)
MUTANTS = [
    ("lamb_m_no_dampening", "+ (1.0 - beta1) * gj;", "+ gj;", 0),
    ("lamb_v_uses_beta1", "double vj = beta2 * (double)v[j] + (1.0 - beta2)",
     "double vj = beta1 * (double)v[j] + (1.0 - beta1)", 0),
    ("lamb_v_abs_not_square", "(gj * gj)", "fabs(gj)", 0),
    ("lamb_c1_exponent_plus_one", "pow(beta1, (double)t)", "pow(beta1, (double)(t + 1))", 0),
    ("lamb_c2_exponent_plus_one", "pow(beta2, (double)t)", "pow(beta2, (double)(t + 1))", 0),
    ("lamb_c1_c2_swapped", "double m_hat = mj / c1;", "double m_hat = mj / c2;", 0),
    ("lamb_no_m_correction", "double m_hat = mj / c1;", "double m_hat = mj;", 0),
    ("lamb_no_v_correction", "double v_hat = vj / c2;", "double v_hat = vj;", 0),
    ("lamb_eps_inside_sqrt", "(sqrt(v_hat) + eps)", "sqrt(v_hat + eps)", 0),
    ("lamb_eps_dropped", "(sqrt(v_hat) + eps)", "(sqrt(v_hat))", 0),
    ("lamb_eps_before_correction", "double r = m_hat / (sqrt(v_hat) + eps);",
     "double r = (mj / (sqrt(vj) + eps)) / c1 * sqrt(c2);", 0),
    ("lamb_lambda_dropped", "u[j] = r + lam * xj;", "u[j] = r;", 0),
    ("lamb_lambda_sign", "u[j] = r + lam * xj;", "u[j] = r - lam * xj;", 0),
    ("lamb_mask_ignored", "double lam = wd ? weight_decay : 0.0;",
     "double lam = weight_decay;", 0),
    ("lamb_norm_of_r", "sum_uu = norm_add(norm, sum_uu, u[j]);",
     "sum_uu = norm_add(norm, sum_uu, r);", 0),
    ("lamb_phi_of_norm_u", "phi(norm_x, gamma_l, gamma_u) / norm_u;",
     "phi(norm_u, gamma_l, gamma_u) / norm_u;", 0),
    ("lamb_not_normalised", "phi(norm_x, gamma_l, gamma_u) / norm_u;",
     "phi(norm_x, gamma_l, gamma_u);", 0),
    ("lamb_update_sign", "(double)x[j] - lr * ratio * u[j]", "(double)x[j] + lr * ratio * u[j]", 0),
    ("lamb_stores_corrected_m", "m[j] = store_f32(mj);", "m[j] = store_f32(m_hat);", 0),
    ("lamb_stores_corrected_v", "v[j] = store_f32(vj);", "v[j] = store_f32(v_hat);", 0),
    ("lamb_zero_norm_not_guarded", "(norm_u == 0.0) ? 0.0 :", "", 0),
    ("phi_no_lower_clamp", "if (p < gamma_l)\n        p = gamma_l;", "", 0),
    ("phi_no_upper_clamp", "if (p > gamma_u)\n        p = gamma_u;", "", 0),
    ("phi_bounds_swapped", "p = gamma_l;\n    if (p > gamma_u)\n        p = gamma_u;",
     "p = gamma_u;\n    if (p > gamma_u)\n        p = gamma_l;", 0),
    ("bf16_wrong_shift", "(uint32_t)bits << 16", "(uint32_t)bits << 15", 0),
    ("lars_no_dampening", "(1.0 - beta1) * (gj + lam * xj)", "(gj + lam * xj)", 0),
    ("lars_lambda_dropped", "(1.0 - beta1) * (gj + lam * xj)", "(1.0 - beta1) * gj", 0),
    ("lars_lambda_after_momentum", "mt[j] = beta1 * (double)m[j] + (1.0 - beta1) * (gj + lam * xj);",
     "mt[j] = beta1 * (double)m[j] + (1.0 - beta1) * gj + lam * xj;", 0),
    ("lars_mask_ignored", "double lam = wd ? weight_decay : 0.0;",
     "double lam = weight_decay;", 1),
    ("lars_no_trust_coef", "trust_coef * phi(norm_x, gamma_l, gamma_u) / norm_m",
     "phi(norm_x, gamma_l, gamma_u) / norm_m", 0),
    ("lars_norm_of_g", "sum_mm = norm_add(norm, sum_mm, mt[j]);",
     "sum_mm = norm_add(norm, sum_mm, gj);", 0),
    ("lars_phi_of_norm_m", "phi(norm_x, gamma_l, gamma_u) / norm_m",
     "phi(norm_m, gamma_l, gamma_u) / norm_m", 0),
    ("lars_update_sign", "(double)x[j] - lr * ratio * mt[j]", "(double)x[j] + lr * ratio * mt[j]", 0),
    ("lars_stores_undamped_m", "m[j] = store_f32(mt[j]);",
     "m[j] = store_f32(mt[j] / (1.0 - beta1));", 0),
    ("nlamb_m_next_power", "double b1_next = pow(beta1, (double)(t + 1));",
     "double b1_next = pow(beta1, (double)t);", 0),
    ("nlamb_m_power_index", "double b1_t = pow(beta1, (double)t);",
     "double b1_t = pow(beta1, (double)(t + 1));", 0),
    ("nlamb_m_drops_gradient_term",
     "double m_hat = beta1 * mj / (1.0 - b1_next) + (1.0 - beta1) * gj / (1.0 - b1_t);",
     "double m_hat = beta1 * mj / (1.0 - b1_next);", 0),
    ("nlamb_m_no_beta_factor",
     "double m_hat = beta1 * mj / (1.0 - b1_next) + (1.0 - beta1) * gj / (1.0 - b1_t);",
     "double m_hat = mj / (1.0 - b1_next) + (1.0 - beta1) * gj / (1.0 - b1_t);", 0),
    ("nlamb_v_no_beta_factor", "v_hat = beta2 * vj / (1.0 - b2_t);", "v_hat = vj / (1.0 - b2_t);", 0),
    ("nnlamb_v_next_power", "double b2_next = pow(beta2, (double)(t + 1));",
     "double b2_next = pow(beta2, (double)t);", 0),
    ("nnlamb_v_drops_gradient_term",
     "v_hat = beta2 * vj / (1.0 - b2_next) + (1.0 - beta2) * (gj * gj) / (1.0 - b2_t);",
     "v_hat = beta2 * vj / (1.0 - b2_next);", 0),
    ("nlamb_flags_swapped", "if (nesterov_v)", "if (!nesterov_v)", 0),
    ("nlamb_mask_ignored", "double lam = wd ? weight_decay : 0.0;", "double lam = weight_decay;", 2),
    ("nlamb_eps_inside_sqrt", "double r = m_hat / (sqrt(v_hat) + eps);",
     "double r = m_hat / sqrt(v_hat + eps);", 1),
    ("lamb_grad_scale_dropped", "double gj = grad_scale * gradient_at(g, g_is_bf16, j);",
     "double gj = gradient_at(g, g_is_bf16, j);", 0),
    ("lars_grad_scale_dropped", "double gj = grad_scale * gradient_at(g, g_is_bf16, j);",
     "double gj = gradient_at(g, g_is_bf16, j);", 1),
    ("nlamb_grad_scale_dropped", "double gj = grad_scale * gradient_at(g, g_is_bf16, j);",
     "double gj = gradient_at(g, g_is_bf16, j);", 2),
    ("l1_squares", "return acc + fabs(a);", "return acc + a * a;", 0),
    ("linf_no_abs", "double b = fabs(a);", "double b = a;", 0),
    ("linf_sums", "return (isnan(b) || b > acc) ? b : acc;", "return acc + b;", 0),
    ("norm_finish_sqrt_always", "return norm == ORACLE_NORM_L2 ? sqrt(acc) : acc;",
     "return sqrt(acc);", 0),
    ("finite_check_in_double", "float p = gj * s;", "double p = (double)gj * 10.0 * (double)s / 10.0;", 0),
    ("finite_check_ignores_nan", "if (!isfinite(p))", "if (isinf(p))", 0),
    ("bf16_round_half_up", "if (low > 0x8000u || (low == 0x8000u && (high & 1u)))",
     "if (low >= 0x8000u)", 0),
    ("bf16_truncate", "            high += 1u;", "            high += 0u;", 0),
    ("bf16_nan_payload", "            out[j] = 0x7fc0;", "            out[j] = 0x7f80;", 0),
    ("lars_zero_norm_not_guarded", "(norm_m == 0.0)\n                       ? 0.0\n                       :", "", 0),
]


def _in_comment(text, pos):
    line = text[text.rfind("\n", 0, pos) + 1:pos].lstrip()
    return line.startswith(("*", "/*", "//"))


def _mutate(text, old, new, occurrence):
    """Replace the ``occurrence``-th appearance of ``old`` in code (not comments)."""
    pos, seen = -1, -1
    while seen < occurrence:
        pos = text.find(old, pos + 1)
        assert pos >= 0, "mutation anchor not found in code: %r" % old
        if not _in_comment(text, pos):
            seen += 1
    return text[:pos] + new + text[pos + len(old):]


@pytest.mark.parametrize("name,old,new,occ", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new, occ):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    with open(oracle.SOURCE) as f:
        text = f.read()
    src = tmp_path / (name + ".c")
    src.write_text(_mutate(text, old, new, occ))
    lib = oracle.build(str(src), str(tmp_path / ("lib" + name + ".so")))
    mutant = oracle.Oracle(lib)
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(mutant)
        except (AssertionError, RuntimeError, FloatingPointError):
            caught.append(pin.__name__)
    assert caught, "no pin catches mutant %s" % name
    os.remove(lib)
