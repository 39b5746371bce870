"""Plausible mistakes planted in a copy of the oracle must fail at least one pin (no GPU).

Each mutant is the oracle source with one textual change (a dropped term, a
wrong budget, a wrong tie rule, a missing forget, ...), compiled on the side.
The pins of ``test_oracle.py`` are then run against it; a mutant that passes
them all means the pins have a blind spot.
"""
import os
import shutil

import pytest

import oracle
import test_oracle as T
import test_oracle_sweep as S

SRC = os.path.join(os.path.dirname(oracle.__file__), "rko.c")

# (name, original text, replacement, which occurrence (0-based) or None for all)
MUTANTS = [
    ("sweep_drops_input_of_later_forwards",
     "int64_t use = (k > s ? (int64_t)c->x[k] : 0) + c->x[k + 1] + c->fn_tmp[k];",
     "int64_t use = c->x[k + 1] + c->fn_tmp[k];", 0),
    ("sweep_drops_temp", "+ c->x[k + 1] + c->fn_tmp[k];\n            sweep_time",
     "+ c->x[k + 1];\n            sweep_time", 0),
    ("case1_rest_budget_ignores_output",
     "rest = get_opt(c, opt, ncells, s + 1, t, m - xbar);",
     "rest = get_opt(c, opt, ncells, s + 1, t, m - c->mem[(int64_t)s * K + o]);", 0),
    ("case1_ignores_backward_temp",
     "if (m < xbar + c->tmp_bwd[(int64_t)s * K + o]) continue;", "", 0),
    ("case1_ignores_forward_temp",
     "if (m < xbar + c->tmp_fwd[(int64_t)s * K + o]) continue;", "", 0),
    ("case2_right_budget_keeps_x_i",
     "get_opt(c, opt, ncells, i, t, m - c->x[i])", "get_opt(c, opt, ncells, i, t, m)", 0),
    ("case2_left_budget_minus_x_i",
     "get_opt(c, opt, ncells, s, i - 1, m)", "get_opt(c, opt, ncells, s, i - 1, m - c->x[i])", 0),
    ("case2_sweep_time_skips_first_forward",
     "sweep_time += c->fn_time[k];", "sweep_time += (k > s) ? c->fn_time[k] : 0;", 1),
    ("case2_split_range_excludes_t",
     "for (int32_t i = s + 1; i <= t; ++i) {\n            int32_t k = i - 1; /* F_k^0",
     "for (int32_t i = s + 1; i < t; ++i) {\n            int32_t k = i - 1; /* F_k^0", 0),
    ("case1_costs_forward_only",
     "int64_t v = (int64_t)c->fwd[(int64_t)s * K + o] + c->bwd[(int64_t)s * K + o] + rest;",
     "int64_t v = (int64_t)c->fwd[(int64_t)s * K + o] + rest;", 0),
    ("tie_prefers_case1", "(v == best && L + o < code)", "(v == best)", 0),
    ("tie_prefers_larger_split", "(v == best && i < code)", "(v == best)", 0),
    ("answer_ignores_x0", "*answer = opt[(int64_t)(M - c->x[0]) * ncells",
     "*answer = opt[(int64_t)(M) * ncells", 0),
    ("build_case1_wrong_budget", "if (t > s) build(c, arg, harg, ncells, s + 1, t, m - xbar, e);",
     "if (t > s) build(c, arg, harg, ncells, s + 1, t, m, e);", 0),
    ("build_forgets_no_x_i", "emit(e, RKO_FREE_X, i, -1);\n", "", 1),
    ("build_keeps_sweep_activations", "emit(e, RKO_FREE_X, k, -1);\n", "", 1),
    ("simulator_forward_ignores_temp",
     "if (used + add + c->tmp_fwd[(int64_t)k * K + o] > pk)\n                pk = used + add + c->tmp_fwd[(int64_t)k * K + o];",
     "if (used + add > pk)\n                pk = used + add;", 0),
    ("simulator_backward_frees_input",
     "used -= (int64_t)c->x[k + 1] + c->mem[(int64_t)k * K + o];",
     "used -= (int64_t)c->x[k] + c->mem[(int64_t)k * K + o];", 0),
    ("min_feasible_drops_x_i",
     "int64_t need = max64(sweep, max64((int64_t)c->x[i] + out[rko_cell(L, i, t)],",
     "int64_t need = max64(sweep, max64((int64_t)out[rko_cell(L, i, t)],", 1),
    # the saving sweep (case 3)
    ("sweep_left_budget_keeps_input", "get_opt(c, opt, ncells, s, i - 1, u - c->x[s])",
     "get_opt(c, opt, ncells, s, i - 1, u)", 0),
    ("sweep_right_budget_keeps_x_i", "get_opt(c, opt, ncells, i, t, u - c->x[i])",
     "get_opt(c, opt, ncells, i, t, u)", 0),
    ("sweep_validity_drops_input", "int64_t use = (int64_t)c->x[k] + c->x[k + 1] + c->fn_tmp[k];",
     "int64_t use = c->x[k + 1] + c->fn_tmp[k];", 0),
    ("sweep_time_skips_first_forward",
     "sweep_time += c->fn_time[k];", "sweep_time += (k > s) ? c->fn_time[k] : 0;", 0),
    ("sweep_costs_no_refwd", "c->refwd[(int64_t)s * K + o] + h;", "h;", 0),
    ("sweep_h_budget_minus_xbar", "hval[(m - mem) * ncells", "hval[(m - xbar) * ncells", 0),
    ("sweep_tie_prefers_sweep", "(v == best && L + K + o < code)", "(v == best)", 0),
    ("sweep_ignores_backward_temp", "if (m < xbar + c->tmp_bwd[(int64_t)s * K + o]) continue;", "", 1),
    ("build_sweep_no_refwd", "emit(e, RKO_REFWD, s, o);\n", "", 0),
    ("build_sweep_left_budget", "build(c, arg, harg, ncells, s + 1, i - 1, u - c->x[s + 1], e);",
     "build(c, arg, harg, ncells, s + 1, i - 1, u, e);", 0),
    ("build_sweep_forgets_no_x_i", "emit(e, RKO_FREE_X, i, -1);\n", "", 0),
    ("build_sweep_keeps_activations", "emit(e, RKO_FREE_X, k, -1);\n", "", 0),
    ("simulator_refwd_ignores_temp",
     "if (used + c->x[k + 1] + c->tmp_fwd[(int64_t)k * K + o] > pk)\n                pk = used + c->x[k + 1] + c->tmp_fwd[(int64_t)k * K + o];",
     "if (used + c->x[k + 1] > pk)\n                pk = used + c->x[k + 1];", 0),
    ("simulator_refwd_is_free", "tm += c->refwd[(int64_t)k * K + o];", "", 0),
    ("min_feasible_sweep_drops_input", "(int64_t)c->x[s] + out[rko_cell(L, s, i - 1)]",
     "out[rko_cell(L, s, i - 1)]", 0),
]


def _mutate(text, old, new, occ):
    assert text.count(old) > occ, f"mutation anchor not found: {old!r}"
    parts = text.split(old)
    return old.join(parts[:occ + 1]) + new + old.join(parts[occ + 1:])


def _pins(lib):
    T.check_worked_example(lib)
    T.check_tie_example(lib)
    T.check_bruteforce(T.tiny_chains(14), lib)
    T.check_inf_pattern(T.random_mid_chains()[:3], lib)
    T.check_store_all(T.random_mid_chains()[:2], lib)
    for ch in T.random_mid_chains()[:3]:
        hi = T.store_all_bound(ch)
        T.check_replay(ch, [hi // 3, hi // 2, hi], lib)
    # the saving sweep
    S.check_sweep_example(lib)
    S.check_bruteforce_sweep(S.tiny_sweep_chains(12), lib)
    S.check_inf_pattern_sweep(S.mid_sweep_chains()[:3], lib)
    S.check_replay_sweep(S.mid_sweep_chains()[:4], lib)


@pytest.mark.parametrize("name,old,new,occ", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new, occ):
    text = open(SRC).read()
    src = tmp_path / "rko_mut.c"
    src.write_text(_mutate(text, old, new, occ))
    shutil.copy(os.path.join(os.path.dirname(SRC), "rko.h"), tmp_path / "rko.h")
    lib = oracle.build_variant(str(src), str(tmp_path / "librko_mut.so"))
    with pytest.raises((AssertionError, ValueError)):
        _pins(lib)


def test_unmutated_source_passes_pins(tmp_path):
    src = tmp_path / "rko_copy.c"
    shutil.copy(SRC, src)
    shutil.copy(os.path.join(os.path.dirname(SRC), "rko.h"), tmp_path / "rko.h")
    _pins(oracle.build_variant(str(src), str(tmp_path / "librko_copy.so")))
