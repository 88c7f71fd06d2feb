"""Every plausible mistake planted in a copy of the oracle's C source must
fail at least one pin (CPU only; the oracle in the tree is untouched).

Each mutant names the passage of the paper, or the reading of it, that the
planted mistake contradicts."""

import os
import subprocess
import tempfile

import pytest

import oracle
import oracle_pins

SRC = open(oracle._SRC).read()

# (name, original text, replacement, which occurrence (0-based) to replace)
MUTANTS = [
    ("ema_weights_swapped_adam", "beta[j] * load(u[j], c->m_dtype, i) + (1.0 - beta[j]) * gh",
     "(1.0 - beta[j]) * load(u[j], c->m_dtype, i) + beta[j] * gh", 0),
    ("ema_weights_swapped_sgdm", "beta[j] * load(u[j], c->m_dtype, i) + (1.0 - beta[j]) * gh",
     "(1.0 - beta[j]) * load(u[j], c->m_dtype, i) + beta[j] * gh", 1),
    ("ema_weights_swapped_adopt", "beta[j] * load(u[j], c->m_dtype, i) + (1.0 - beta[j]) * gn",
     "(1.0 - beta[j]) * load(u[j], c->m_dtype, i) + beta[j] * gn", 0),
    ("beta_index_fixed_to_first", "beta[j] * load(u[j], c->m_dtype, i) + (1.0 - beta[j]) * gh",
     "beta[0] * load(u[j], c->m_dtype, i) + (1.0 - beta[0]) * gh", 0),
    ("omega_index_fixed_to_first", "num += omega[j] * (uj / bc[j]);", "num += omega[0] * (uj / bc[j]);", 0),
    ("gradient_term_dropped_adam", "double num = g_weight * gh;", "double num = 0.0 * gh;", 0),
    ("gradient_weight_sign", "const double g_weight = 1.0 - omega_sum;",
     "const double g_weight = omega_sum - 1.0;", 0),
    ("gradient_weight_is_one", "const double g_weight = 1.0 - omega_sum;",
     "const double g_weight = 1.0;", 0),
    ("bias_correction_step_off_by_one", "bc[j] = 1.0 - pow(beta[j], (double)s);",
     "bc[j] = 1.0 - pow(beta[j], (double)(s + 1));", 0),
    ("second_moment_uncorrected", "bc2 = 1.0 - pow(beta2, (double)s);", "bc2 = 1.0;", 0),
    ("eps_inside_sqrt_adam", "sqrt(vv / bc2) + eps", "sqrt(vv / bc2 + eps)", 0),
    ("eps_inside_sqrt_adopt", "gn = graw / (sqrt(vv) + eps);", "gn = graw / sqrt(vv + eps);", 0),
    ("adam_v_uses_raw_gradient", "(1.0 - beta2) * gh * gh", "(1.0 - beta2) * graw * graw", 0),
    ("update_sign_adam", "load(x, c->x_dtype, i) - eta * delta", "load(x, c->x_dtype, i) + eta * delta", 0),
    ("update_sign_sgdm", "load(x, c->x_dtype, i) - eta * delta", "load(x, c->x_dtype, i) + eta * delta", 2),
    ("sgdm_gradient_term_unclipped", "double delta = g_weight * gh;", "double delta = g_weight * graw;", 0),
    ("adopt_prev_uses_new_v", "gn = graw / (sqrt(vv) + eps);\n          vv = beta2 * vv + (1.0 - beta2) * graw * graw;",
     "vv = beta2 * vv + (1.0 - beta2) * graw * graw;\n          gn = graw / (sqrt(vv) + eps);", 0),
    ("adopt_first_step_updates_x", "store(v, c->m_dtype, i, graw * graw);\n            continue;",
     "store(v, c->m_dtype, i, graw * graw);\n            vv = graw * graw;\n            gn = graw / (sqrt(vv) + eps);", 0),
    ("adopt_no_clamp", "if (cc > 0.0) gn = gn > cc", "if (cc < 0.0) gn = gn > cc", 0),
    ("adopt_gradient_term_dropped", "double delta = g_weight * gn;", "double delta = 0.0 * gn;", 0),
    ("schedule_phase_shift", "if (period_x > 0 && s % period_x == 0)",
     "if (period_x > 0 && (s - 1) % period_x == 0)", 0),
    ("schedule_u_bit_off_by_one", "mask |= 1u << (j + 1);", "mask |= 1u << j;", 0),
    ("schedule_v_ignores_form", "if (has_v && period_v > 0", "if (period_v > 0", 0),
    ("schedule_only_first_moment", "if (period_u[j] > 0 && s % period_u[j] == 0)",
     "if (j == 0 && period_u[j] > 0 && s % period_u[j] == 0)", 0),
    ("mean_divides_by_k_minus_one", "const double mean = acc / (double)K;",
     "const double mean = acc / (double)(K > 1 ? K - 1 : 1);", 0),
    ("mean_written_to_first_row_only", "for (int64_t m = 0; m < K; ++m) store(state, dtype, m * P + p, mean);",
     "for (int64_t m = 0; m < 1; ++m) store(state, dtype, m * P + p, mean);", 0),
    ("mean_skips_last_worker", "for (int64_t m = 0; m < K; ++m) acc += load(state, dtype, m * P + p);",
     "for (int64_t m = 0; m + 1 < K; ++m) acc += load(state, dtype, m * P + p);", 0),
    ("clip_scale_not_capped", "return c < 1.0 ? c : 1.0;", "return c;", 0),
    ("clip_norm_is_l1", "acc += a * a;", "acc += fabs(a);", 0),
    ("bf16_truncates", "ldexp(nearbyint(ldexp(a, -q)), q)", "ldexp(trunc(ldexp(a, -q)), q)", 0),
    ("bf16_ties_away", "ldexp(nearbyint(ldexp(a, -q)), q)", "ldexp(round(ldexp(a, -q)), q)", 0),
    ("bf16_no_subnormals", "if (q < -133) q = -133;", "if (q < -126) q = -126;", 0),
    ("prob_step_omega_index", "for (int32_t j = 0; j < n; ++j) delta += omega[j] * load(u[j], c->m_dtype, i);",
     "for (int32_t j = 0; j < n; ++j) delta += omega[0] * load(u[j], c->m_dtype, i);", 0),
    ("prob_step_ema_weights_swapped",
     "store(u[j], c->m_dtype, i, beta[j] * load(u[j], c->m_dtype, i) + (1.0 - beta[j]) * gh);",
     "store(u[j], c->m_dtype, i, (1.0 - beta[j]) * load(u[j], c->m_dtype, i) + beta[j] * gh);", 0),
    ("prob_step_u_mean_skips_last_worker",
     "for (int64_t m = 0; m < K; ++m) acc += load(u[j], c->m_dtype, m * P + p);",
     "for (int64_t m = 0; m + 1 < K; ++m) acc += load(u[j], c->m_dtype, m * P + p);", 0),
    ("prob_step_no_x_average", "    if (mask & 1u) {\n      double acc = 0.0;",
     "    if (mask & 0u) {\n      double acc = 0.0;", 0),
    ("outer_plain_momentum", "(double)xo[p] - lr * (d + m_ * (double)b[p]);", "(double)xo[p] - lr * ((double)b[p]);", 0),
    ("outer_gradient_sign", "const double d = (double)xo[p] - xbar;", "const double d = xbar - (double)xo[p];", 0),
    ("outer_no_momentum", "const double bn = m_ * (double)b[p] + d;", "const double bn = d;", 0),
    ("stats_variance_not_centered", "out[1] += (c - cbar) * (c - cbar);", "out[1] += c * c;", 0),
    ("stats_pseudo_gradient_sign", "cbar += xo ? (double)xo[p] - v : v;", "cbar += xo ? v - (double)xo[p] : v;", 0),
    ("stats_dot_uses_norm", "out[4 + K + m] += c * cbar;", "out[4 + K + m] += c * c;", 0),
    ("f32_store_truncates", "float f = (float)a;\n    ((float*)p)[i] = f;",
     "float f = (float)a;\n    if ((double)f > a && f > 0) f = nextafterf(f, 0.0f);\n    ((float*)p)[i] = f;", 0),
]


def _mutate(name, old, new, occ):
    parts = SRC.split(old)
    assert len(parts) > occ + 1, f"{name}: target text not found"
    return old.join(parts[: occ + 1]) + new + old.join(parts[occ + 1:])


@pytest.fixture(scope="module")
def workdir():
    with tempfile.TemporaryDirectory() as d:
        yield d
    oracle.use_library(oracle._LIB)


@pytest.mark.parametrize("mutant", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(mutant, workdir):
    name, old, new, occ = mutant
    src = os.path.join(workdir, f"{name}.c")
    so = os.path.join(workdir, f"{name}.so")
    with open(src, "w") as f:
        f.write(_mutate(name, old, new, occ))
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared",
                    *(oracle.SAN_FLAGS if oracle.SANITIZE else []), "-o", so, src, "-lm"], check=True)
    oracle.use_library(so)
    try:
        for pin in oracle_pins.ALL_PINS:
            try:
                pin()
            except (AssertionError, FloatingPointError, ValueError, ZeroDivisionError):
                return  # caught
        pytest.fail(f"mutant {name} passed every pin")
    finally:
        oracle.use_library(oracle._LIB)
