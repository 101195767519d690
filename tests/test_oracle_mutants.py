"""Planted mistakes in the CPU oracle must be caught by its pins.

Each mutant is a copy of oracle/lif_oracle.c with one plausible mistake (a
dropped term, a wrong sign, a shifted index, a transposed layout, a different
reading of the tie rule or of the reset).  It is compiled on the CPU into a
temporary library, every pin of tests/oracle_pins.py is run against it, and at
least one pin has to fail.  CPU only.
"""
import os
import shutil

import pytest

import oracle
from tests import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "lif_oracle.c")

MUTANTS = {
    "tie_is_no_spike": ("yt = (vt - th >= 0.0f) ? 1 : 0;", "yt = (vt - th > 0.0f) ? 1 : 0;"),
    "reset_value_decayed": ("vt = yt ? rest + xt : k * vt + xt;", "vt = yt ? k * rest + xt : k * vt + xt;"),
    "reset_ignores_v_rest": ("vt = yt ? rest + xt : k * vt + xt;", "vt = yt ? xt : k * vt + xt;"),
    "no_leak": ("vt = yt ? rest + xt : k * vt + xt;", "vt = yt ? rest + xt : vt + xt;"),
    "reset_never": ("vt = yt ? rest + xt : k * vt + xt;", "vt = k * vt + xt;"),
    "soft_subtract_after_leak": ("vt = k * w + xt;", "vt = k * vt - (yt ? th : 0.0f) + xt;"),
    "soft_no_subtract": ("float w = yt ? vt - th : vt;", "float w = vt;"),
    "initial_membrane_zero": ("float vt = v_init ? v_init[n] : rest;", "float vt = v_init ? v_init[n] : 0.0f;"),
    "initial_spike_one": ("int yt = y_init ? (y_init[n] != 0) : 0;", "int yt = y_init ? (y_init[n] != 0) : 1;"),
    "input_one_step_late": ("const float xt = x[t * N + n];", "const float xt = x[(t > 0 ? t - 1 : 0) * N + n];"),
    "layout_transposed": ("const float xt = x[t * N + n];", "const float xt = x[n * T + t];"),
    "surrogate_at_v_not_v_minus_th": ("surrogate(alpha, vt - th)", "surrogate(alpha, vt)"),
    "surrogate_drops_alpha": ("return alpha * e / ((1.0 + e) * (1.0 + e));", "return e / ((1.0 + e) * (1.0 + e));"),
    "surrogate_not_squared": ("return alpha * e / ((1.0 + e) * (1.0 + e));", "return alpha * e / (1.0 + e);"),
    "reset_term_sign": ("(rest - k * vt) * d;", "(k * vt - rest) * d;"),
    "reset_detached": ("D = k * (1.0 - (double)y[i]) + (rest - k * vt) * d;",
                       "D = k * (1.0 - (double)y[i]);"),
    "reset_gate_dropped": ("D = k * (1.0 - (double)y[i]) + (rest - k * vt) * d;",
                           "D = k + (rest - k * vt) * d;"),
    "soft_backward_sign": ("D = k * (1.0 - th * d);", "D = k * (1.0 + th * d);"),
    "soft_backward_detached": ("D = k * (1.0 - th * d);", "D = k;"),
    "recurrence_factor_k_only": ("const double g = gy[i] * d + D * g_after;",
                                 "const double g = gy[i] * d + k * g_after;"),
    "direct_term_dropped": ("const double g = gy[i] * d + D * g_after;",
                            "const double g = gy[i] + D * g_after;"),
    "terminal_gradient_one": ("double g_after = g_next ? g_next[n] : 0.0;",
                              "double g_after = g_next ? g_next[n] : 1.0;"),
    "gain_glue_wrong_index": ("x_next[i] = gain[f] * (float)y[i];", "x_next[i] = gain[b % F] * (float)y[i];"),
    # the stack of layers joined by a gain
    "stack_forward_first_gain_everywhere": ("gains + l * F, xs + (l + 1) * TN);", "gains, xs + (l + 1) * TN);"),
    "stack_forward_x_to_every_layer": ("lif_oracle_forward(p, T, B * F, xs + l * TN,",
                                       "lif_oracle_forward(p, T, B * F, x,"),
    "stack_backward_gain_of_other_layer": ("gains + l * F, h_g,", "gains + (L - 2 - l) * F, h_g,"),
    "stack_backward_gain_index": ("const double a = (double)gain[f];", "const double a = (double)gain[b % F];"),
    "stack_backward_gain_dropped": ("gy[i] = a * gx_next[i];", "gy[i] = gx_next[i];"),
    "stack_backward_ignores_layer_above": ("lif_oracle_backward(p, T, N, v + o, y + o, h_g, h_err,",
                                           "lif_oracle_backward(p, T, N, v + o, y + o, gy, h_err,"),
    "stack_backward_budget_as_gradient": ("lif_oracle_gain_backward(T, B, F, gx + o + TN,",
                                          "lif_oracle_gain_backward(T, B, F, gx_err + o + TN,"),
    "stack_backward_layer0_membranes": ("lif_oracle_backward(p, T, N, v + o, y + o, h_g,",
                                        "lif_oracle_backward(p, T, N, v, y, h_g,"),
    # the error budgets
    "budget_without_condition_number": ("d * (1.0 + alpha * fabs(vt - th))", "d"),
    "budget_propagated_by_term_magnitudes": ("fabs(D) * e_after;", "m * e_after;"),
    "budget_without_factor_rounding": ("+ m * fabs(g_after) +", "+"),
    "budget_without_direct_term": ("fabs(gy[i]) * dc +", ""),
    "budget_rounding_not_carried": ("const double r = (gy_rnd ? gy_rnd[i] * d : 0.0) + fabs(D) * r_after;",
                                    "const double r = gy_rnd ? gy_rnd[i] * d : 0.0;"),
    "budget_handoff_rounding_ignored": ("h_rnd[i] += fabs(h_g[i]);", "h_rnd[i] += 0.0;"),
}


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    d = tmp_path_factory.mktemp("oracle_mutants")
    shutil.copy(os.path.join(os.path.dirname(SRC), "lif_oracle.h"), d)
    return d


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(mutant_dir, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(old, new)
    c_path = os.path.join(mutant_dir, f"{name}.c")
    with open(c_path, "w") as f:
        f.write(mutated)
    so = oracle.build(c_path, os.path.join(mutant_dir, f"lib{name}.so"))
    lib = oracle.load(so)
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(lib)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake {name}"
