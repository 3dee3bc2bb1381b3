"""Planted mistakes in copies of the oracle must each fail some pin.

Every mutation below is a plausible slip (a dropped term, a wrong sign, a
wrong index, a misplaced constant).  Each is applied to a copy of oracle.c in
a temporary directory, compiled, and run through the pins; the test passes
only if some pin rejects it.  The real oracle is never modified.
"""
import os
import shutil

import pytest

import oracle
import pins

MUTATIONS = {
    "decay_dropped": ("double p1 = p - (hp->lr * hp->weight_decay) * p;", "double p1 = p;"),
    "decay_sign": ("double p1 = p - (hp->lr", "double p1 = p + (hp->lr"),
    "decay_uses_lr_only": ("(hp->lr * hp->weight_decay) * p", "(hp->weight_decay) * p"),
    "m_history_dropped": ("double m1 = hp->beta1 * m +", "double m1 = 0.0 * m +"),
    "m_wrong_coef": ("(1.0 - hp->beta1) * g;", "hp->beta1 * g;"),
    "v_not_squared": ("(1.0 - hp->beta2) * (g * g)", "(1.0 - hp->beta2) * fabs(g)"),
    "v_uses_beta1": ("double v1 = hp->beta2 * v", "double v1 = hp->beta1 * v"),
    "eps_inside_sqrt": ("(sqrt(v_hat) + hp->eps)", "sqrt(v_hat + hp->eps)"),
    "no_bias_correction_1": ("double m_hat = m1 / bc1;", "double m_hat = m1;"),
    "no_bias_correction_2": ("double v_hat = v1 / bc2;", "double v_hat = v1;"),
    "step_sign": ("*po = p1 - hp->lr", "*po = p1 + hp->lr"),
    "bias_uses_step_minus_1": ("pow(hp->beta1, (double)hp->step)", "pow(hp->beta1, (double)(hp->step + 1))"),
    "mean_not_divided": ("if (exact && (R & (R - 1)) == 0)\n        return (float)(s / (double)R);",
                         "if (exact && (R & (R - 1)) == 0)\n        return (float)s;"),
    "mean_rank0_only": ("double x = (double)orc_f32_from_bf16(grads[r][i]);",
                        "double x = (double)orc_f32_from_bf16(grads[0][i]);"),
    "mean_fp32_sum": ("        s = t;\n", "        s = (float)t;\n"),
    "mean_double_rounded": ("if (exact && (R & (R - 1)) == 0)", "if (1)"),
    "mean_inexact_sum_trusted": ("if (exact && (R & (R - 1)) == 0)", "if ((R & (R - 1)) == 0)"),
    "mean_exact_not_divided": ("fix_div_small(&pos, (uint32_t)R);", "fix_div_small(&pos, 1u);"),
    "mean_exact_no_remainder": ("int sticky = rem != 0 || fix_any_below(&pos, lsb - 1);",
                                "int sticky = fix_any_below(&pos, lsb - 1);"),
    "mean_exact_truncates": ("        ++mant; /* may become 2^24", "        (void)0; /* may become 2^24"),
    "mean_exact_sign_lost": ("return (float)(sign ? -mag : mag);", "return (float)mag;"),
    "mean_exact_negatives_ignored": ("fix_add_shifted((b & 0x8000u) ? &neg : &pos, M, k - MEAN_E0);",
                                     "fix_add_shifted(&pos, M, k - MEAN_E0);"),
    "mean_exact_subnormal_bit": ("uint64_t M = e ? (0x80u | f) : f;", "uint64_t M = 0x80u | f;"),
    "mean_exact_high_part_dropped": ("        fix_add_at(a, k + 1, m >> (64 - s));", "        (void)0;"),
    "mean_exact_subnormal_grid": ("-149 - MEAN_E0", "-150 - MEAN_E0"),
    "mean_exact_borrow_dropped": ("borrow = (x < y) || (x == y && borrow);", "borrow = (x < y);"),
    "norm_no_sqrt": ("    return sqrt(acc_round(&total));", "    return acc_round(&total);"),
    "norm_first_segment_only": ("for (int32_t s = 0; s < n_segs; ++s) {\n        const uint16_t *const *g = segs[s].grads;",
                                "for (int32_t s = 0; s < 1; ++s) {\n        const uint16_t *const *g = segs[s].grads;"),
    "norm_skips_last_element": ("            for (int64_t i = 0; i < n; ++i) {\n                double gb",
                                "            for (int64_t i = 0; i < n - 1; ++i) {\n                double gb"),
    "acc_no_carry": ("        v = a->limb[k] < old; /* carry */", "        v = 0;"),
    "acc_round_no_sticky": ("(acc_any_below(a, lsb - 1) || (mant & 1u))", "(mant & 1u)"),
    "acc_round_truncates": ("        ++mant; /* may become 2^53, still exact */", "        (void)0;"),
    "acc_high_part_dropped": ("        acc_add_at(a, k + 1, m >> (64 - s));", "        (void)0;"),
    "acc_implicit_bit_missing": ("        m |= 1ull << 52;", "        (void)0;"),
    "acc_merge_without_carry": ("    for (int k = 0; k < ACC_LIMBS; ++k)\n        acc_add_at(a, k, b->limb[k]);",
                                "    for (int k = 0; k < ACC_LIMBS; ++k)\n        a->limb[k] += b->limb[k];"),
    "clip_uncapped": ("return c < 1.0 ? c : 1.0;", "return c;"),
    "clip_no_guard": ("max_grad_norm / (norm + 1e-6)", "max_grad_norm / norm"),
    "clip_applied_to_square": ("(double)g_bar * c, hp,", "(double)g_bar * c * c, hp,"),
    "nonfinite_not_skipped": ("if (!isfinite(norm))\n        return ORC_NONFINITE;", ""),
    "bf16_ties_odd": ("pick = ((lo >> 16) & 1u) ? hi : lo;", "pick = ((lo >> 16) & 1u) ? lo : hi;"),
    "bf16_truncates": ("if (dlo < dhi)\n        pick = lo;", "if (1)\n        pick = lo;"),
    "bf16_nan_not_quiet": ("return (uint16_t)((u >> 16) | 0x0040u);", "return (uint16_t)(u >> 16);"),
    "bf16_no_overflow_to_inf": ("ldexp(1.0, 128)", "ldexp(1.0, 200)"),
    "route_gbar_not_rounded": ("return gbar_bf16 ? orc_f32_from_bf16(orc_bf16_from_f32(g_bar)) : g_bar;",
                               "return g_bar;"),
    "route_gbar_truncated": ("return gbar_bf16 ? orc_f32_from_bf16(orc_bf16_from_f32(g_bar)) : g_bar;",
                             "uint32_t u_;\n    memcpy(&u_, &g_bar, 4);\n"
                             "    return gbar_bf16 ? orc_f32_from_bf16((uint16_t)(u_ >> 16)) : g_bar;"),
    "route_points_not_rounded": ("float g_bar = update_gradient(orc_mean_grad(rows, R, 0), gbar_bf16);",
                                 "float g_bar = orc_mean_grad(rows, R, 0);"),
    "param_from_unrounded": ("*pb = orc_bf16_from_f32(*p);", "*pb = orc_bf16_from_f32((float)(po + 1e-9));"),
}

# cheap pins first so that most mutants are rejected quickly
ORDER = ["pin_bf16_special_values", "pin_mean_closed_forms", "pin_norm_constant",
         "pin_exact_sum_ties_and_carries", "pin_exact_sum_vs_fsum",
         "pin_clip_coef", "pin_first_step_sign", "pin_zero_gradient", "pin_sign_descent",
         "pin_lr_zero", "pin_identical_ranks", "pin_clip_noop", "pin_nonfinite",
         "pin_param_is_bf16_of_master", "pin_mean_vs_fraction", "pin_mean_exact_quotient", "pin_norm_vs_torch",
         "pin_adamw_f64_vs_torch", "pin_bf16_random_vs_torch", "pin_bf16_gradient_route",
         "pin_step_vs_torch", "pin_update_given_clip_equals_step",
         "pin_brute_force"]


def test_order_covers_all_pins():
    assert sorted(ORDER) == sorted(p.__name__ for p in pins.ALL_PINS)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutant_is_rejected(name, tmp_path):
    here = os.path.dirname(oracle.__file__)
    src = open(os.path.join(here, "oracle.c")).read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, "mutation anchor not found exactly once"
    shutil.copy(os.path.join(here, "oracle.h"), tmp_path / "oracle.h")
    (tmp_path / "oracle.c").write_text(src.replace(old, new))
    lib = oracle.load(oracle.build(src=str(tmp_path / "oracle.c"),
                                   out=str(tmp_path / "liboracle_mutant.so")))
    failed_by = None
    for pname in ORDER:
        try:
            getattr(pins, pname)(lib)
        except AssertionError:
            failed_by = pname
            break
    assert failed_by is not None, f"mutation {name} passed every pin"
