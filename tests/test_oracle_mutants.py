"""The oracle's pins have teeth: each mutant below plants one plausible
mistake in a copy of the oracle's C source (a dropped term, a wrong sign,
swapped operands, a wrong rounding or overflow rule, a wrong order), builds
it with gcc, and at least one pin of tests/test_oracle_pins.py must fail
against it.  CPU only.  The mistakes are planted in the oracle, never in the
HIP path.
"""
import os

import numpy as np
import pytest

import oracle
import test_oracle_pins as P

# name -> (text in disdp_oracle.c, replacement)
MUTANTS = {
    "moment_sign": ("float mi = b1 * *m + omb1 * g;", "float mi = b1 * *m - omb1 * g;"),
    "drop_eps": ("float d = sqrtf(vh) + eps;", "float d = sqrtf(vh);"),
    "eps_inside_root": ("float d = sqrtf(vh) + eps;", "float d = sqrtf(vh + eps);"),
    "swap_bias_corrections": ("float mh = mi / bc1;\n    float vh = vi / bc2;",
                              "float mh = mi / bc2;\n    float vh = vi / bc1;"),
    "no_second_bias_correction": ("float vh = vi / bc2;", "float vh = vi;"),
    "no_decay": ("float pi = *p * decay - lr * upd;", "float pi = *p - lr * upd;"),
    "v_from_g_not_g2": ("float gg = g * g;", "float gg = g;"),
    "swap_betas": ("float mi = b1 * *m + omb1 * g;", "float mi = b2 * *m + omb2 * g;"),
    "no_grad_scale": ("float g = agg * grad_scale;", "float g = agg;"),
    "drop_first_worker": ("float acc = load_grad(g[0], gdtype, i);", "float acc = 0.0f;"),
    "reverse_worker_order": (
        "float acc = load_grad(g[0], gdtype, i);\n        for (int w = 1; w < W; ++w)\n"
        "            acc = acc + load_grad(g[w], gdtype, i);",
        "float acc = load_grad(g[W - 1], gdtype, i);\n        for (int w = W - 2; w >= 0; --w)\n"
        "            acc = acc + load_grad(g[w], gdtype, i);"),
    "quantise_truncates": ("float r = nearbyintf(y);", "float r = truncf(y);"),
    "quantise_rounds_half_away": ("float r = nearbyintf(y);", "float r = roundf(y);"),
    "int32_sum_wraps": (
        "s += (int64_t)contribution_q(g[w], gdtype, i, k);",
        "s = (int32_t)((uint32_t)s + (uint32_t)contribution_q(g[w], gdtype, i, k));"),
    "nan_quantises_to_one": ("if (y != y)\n        return 0;", "if (y != y)\n        return 1;"),
    "dequantise_wrong_scale": ("agg_f32[i] = (float)a * ldexpf(1.0f, -k);",
                               "agg_f32[i] = (float)a * ldexpf(1.0f, -k + 1);"),
    "int32_contribution_requantised": (
        "return ((const int32_t *)buf)[i];",
        "return oracle_quantize((float)((const int32_t *)buf)[i], k);"),
    "quantise_array_wrong_scale": (
        "out[i] = oracle_quantize(load_grad(g, gdtype, i), k);",
        "out[i] = oracle_quantize(load_grad(g, gdtype, i), k + 1);"),
    "bf16_truncates": ("return (uint16_t)((u + 0x7fffu + lsb) >> 16);",
                       "return (uint16_t)(u >> 16);"),
    "bf16_ties_away": ("return (uint16_t)((u + 0x7fffu + lsb) >> 16);",
                       "return (uint16_t)((u + 0x8000u) >> 16);"),
    "bias_correction_off_by_one": (
        "out[4] = (float)(1.0 - pow((double)beta1, (double)t));",
        "out[4] = (float)(1.0 - pow((double)beta1, (double)(t + 1)));"),
    "decay_sign": ("out[6] = (float)(1.0 - (double)lr * (double)wd);",
                   "out[6] = (float)(1.0 + (double)lr * (double)wd);"),
    "fused_skips_aggregate_output": ("if (agg_f32)\n            agg_f32[i] = a;\n        adamw_element",
                                     "adamw_element"),
}

# the pins run against each mutant, cheapest first; the first to fail ends it
PINS = [
    ("order", P.test_aggregate_order_is_worker_0_first),
    ("identical", lambda: P.test_aggregate_identical_contributions_sum_to_W_g(8)),
    ("first_step", P.test_adamw_first_step_closed_form),
    ("zero_grad", P.test_adamw_zero_gradient_is_pure_decoupled_decay),
    ("scalars", lambda: P.test_scalars_bias_corrections(0.9, 0.95)),
    ("nan_q", P.test_quantize_nan_is_zero),
    ("bf16_ties", P.test_bf16_rne_tie_cases_by_hand),
    ("bf16_torch", P.test_bf16_rne_matches_torch_including_ties),
    ("quantise", lambda: P.test_quantize_matches_exact_rational(0)),
    ("fixed_exact", lambda: P.test_aggregate_fixed_matches_exact(3, 24)),
    ("int32_sum", P.test_aggregate_fixed_of_int32_contributions_is_the_exact_sum),
    ("quantise_array", lambda: P.test_quantize_array_matches_exact_rational("f32", 24)),
    ("composition", lambda: P.test_fused_is_aggregate_then_adamw(4, "f32", oracle.AGG_FP32)),
    ("running_bound", lambda: P.test_adamw_within_running_error_bound_of_exact(3, dict(P.HP))),
    ("torch_adamw", P.test_adamw_matches_torch_adamw),
]


def _run_pins():
    """Name of the first pin that fails, or None."""
    for name, pin in PINS:
        try:
            pin()
        except AssertionError:
            return name
    return None


def test_every_pin_passes_on_the_real_oracle():
    assert _run_pins() is None


def test_every_mutation_site_exists_in_the_source():
    src = oracle.source()
    for name, (old, _new) in MUTANTS.items():
        assert src.count(old) == 1, name


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught_by_a_pin(name, tmp_path):
    old, new = MUTANTS[name]
    path = oracle.build_source(oracle.source().replace(old, new),
                               os.path.join(tmp_path, f"liboracle_{name}.so"))
    with oracle.using(oracle.load_library(path)):
        caught_by = _run_pins()
    assert caught_by is not None, f"no pin fails on mutant {name}"
