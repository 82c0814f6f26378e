"""Plant plausible mistakes in a copy of the oracle (on the CPU) and check
that the pin battery catches every one of them, while the unmodified oracle
passes.  Each mutant is compiled to a temporary library and exercised in a
child process so that a crashing mutant cannot take the test run down."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "esp_oracle.c")

MUTANTS = {
    "rent_drops_a_term": ("for (r = 1; r < p->R; r++) rent", "for (r = 2; r < p->R; r++) rent"),
    "rent_wrong_price": ("rent = rent + (double)d[r] * lam[r];", "rent = rent + (double)d[r] * lam[0];"),
    "score_sign": ("s = (double)util_of(p, b)[e] - rent;", "s = (double)util_of(p, b)[e] + rent;"),
    "switch_sign": ("if (cur >= 0 && k != cur) s = s - p->switch_cost[b];",
                    "if (cur >= 0 && k != cur) s = s + p->switch_cost[b];"),
    "switch_on_current": ("if (cur >= 0 && k != cur) s = s - p->switch_cost[b];",
                          "if (cur >= 0 && k == cur) s = s - p->switch_cost[b];"),
    "penalty_dropped": ("if (p->penalty != NULL) s = s - (double)p->penalty[(int64_t)b * p->nnz + e];", ";"),
    "penalty_wrong_entry": ("if (p->penalty != NULL) s = s - (double)p->penalty[(int64_t)b * p->nnz + e];",
                            "if (p->penalty != NULL) s = s - (double)p->penalty[(int64_t)b * p->nnz + p->offsets[j]];"),
    "ties_to_highest": ("if (best_k < 0 || s > best)", "if (best_k < 0 || s >= best)"),
    "update_sign": ("double g = U[r] - C[r];", "double g = C[r] - U[r];"),
    "no_projection": ("lam[r] = (x > 0.0) ? x : 0.0;", "lam[r] = x;"),
    "negative_zero": ("lam[r] = (x > 0.0) ? x : 0.0;", "lam[r] = (x > 0.0) ? x : -0.0;"),
    "t_zero_based": ("return eta0 / sqrt((double)t);", "return eta0 / sqrt((double)(t + 1));"),
    "rule_swapped": ("if (rule == ORC_STEP_INV_SQRT)", "if (rule != ORC_STEP_INV_SQRT)"),
    "demand_transposed": ("acc_add_f32(&a, d[(p->offsets[j] + choice[j]) * p->R + r]);",
                          "acc_add_f32(&a, d[r * p->nnz + p->offsets[j] + choice[j]]);"),
    "demand_first_config": ("acc_add_f32(&a, d[(p->offsets[j] + choice[j]) * p->R + r]);",
                            "acc_add_f32(&a, d[(p->offsets[j]) * p->R + r]);"),
    "round_half_up": ("if (guard && (sticky || (m & 1u))) m += 1;", "if (guard) m += 1;"),
    "truncating_sum": ("if (guard && (sticky || (m & 1u))) m += 1;", ";"),
    "dual_drops_capacity": ("v = v + lam[r] * p->capacity[(int64_t)b * p->R + r];", ";"),
    "select_skips_last": ("for (e = lo; e < hi; e++) {", "for (e = lo; e + 1 < hi; e++) {"),
    "ceff_max_not_min": ("if (!have || v < m) { m = v; have = 1; }", "if (!have || v > m) { m = v; have = 1; }"),
    "ceff_gamma_dropped": ("g = gamma * S;", "g = S;"),
    "ceff_sign": ("C_eff[r] = C[r] - g;", "C_eff[r] = C[r] + g;"),
    "ceff_queue_ignored": ("if (queued != NULL && queued[j] == 0) continue;", ";"),
    "ceff_mask_ignored": ("if (!entry_allowed(q, b, e)) continue;", ";"),
    "ceff_first_config": ("v = d[e * q->R + r];", "v = d[q->offsets[j] * q->R + r];"),
    "bp_last_fit": ("for (h = 0; h < m->G && found < g; h++)", "for (h = m->G - 1; h >= 0 && found < g; h--)"),
    "bp_ignores_compute": ("mem[h] >= need_m && sm[h] >= need_s", "mem[h] >= need_m"),
    "bp_share_not_divided": ("need_m = (double)d[e * p->R + m->r_mem] / gv;", "need_m = (double)d[e * p->R + m->r_mem];"),
    "iac_wrong_pressure": ("sxy = (double)sa[ex] * (double)pb[ey];", "sxy = (double)sa[ex] * (double)pb[ex];"),
    "iac_no_clamp": ("if (add > m->beta_max) add = m->beta_max;", ";"),
    "iac_and_not_or": ("if (ox > 0.0 || oy > 0.0) V++;", "if (ox > 0.0 && oy > 0.0) V++;"),
    "gamma_not_reset": ("for (e = 0; e < p->nnz; e++) penalty[e] = 0.0f;", ";"),
    "penalty_no_kappa": ("penalty[e] = (float)((double)penalty[e] + m->kappa * inc[j]);",
                         "penalty[e] = (float)((double)penalty[e] + inc[j]);"),
    "rounds_no_break": ("if (V == 0) break;", ";"),
    "nn_abs_not_square": ("acc = x * x;", "acc = fabs(x);"),
    "nn_drops_last_dim": ("for (r = 1; r < p->R; r++) {\n            x = (double)q[r]",
                          "for (r = 1; r + 1 < p->R; r++) {\n            x = (double)q[r]"),
    "nn_ties_highest": ("if (best_k < 0 || acc < best)", "if (best_k < 0 || acc <= best)"),
    "nn_mask_ignored": ("if (!entry_allowed(p, b, e)) continue;\n        x = (double)q[0]",
                        "x = (double)q[0]"),
    "nn_wrong_dim": ("x = (double)q[r] - (double)d[e * p->R + r];", "x = (double)q[r] - (double)d[e * p->R];"),
    "nn_estimate_first": ("util_of(p, b)[p->offsets[family[i]] + c]", "util_of(p, b)[p->offsets[family[i]]]"),
    "stop_post_update_scale": ("double scale = prev[r] > 1.0 ? prev[r] : 1.0;",
                               "double scale = lb[r] > 1.0 ? lb[r] : 1.0;"),
    "stop_strict": ("if (!(diff <= tol * scale)) conv = 0;", "if (!(diff < tol * scale)) conv = 0;"),
    "stop_absolute": ("double scale = prev[r] > 1.0 ? prev[r] : 1.0;", "double scale = 1.0;"),
    "stop_no_unit_floor": ("double scale = prev[r] > 1.0 ? prev[r] : 1.0;", "double scale = prev[r];"),
    "stop_any_resource": ("if (!(diff <= tol * scale)) conv = 0;\n                }\n                if (conv) break;",
                          "if (diff <= tol * scale) conv = 2;\n                }\n                if (conv == 2) break;"),
    "stop_step_not_change": ("double diff = fabs(lb[r] - prev[r]);", "double diff = fabs(eta * (U[r] - Cb[r]));"),
    "stop_never": ("if (conv) break;", ";"),
    "stop_count_off_by_one": ("done = i + 1;", "done = i;"),
    "ceff_whole_config": ("if (!have || v < m) { m = v; have = 1; }",
                          "if (!have || d[e * q->R] < d[(q->offsets[j]) * q->R]) { m = v; have = 1; }"),
}


def _build(tmp_path, name, text):
    src = tmp_path / f"{name}.c"
    src.write_text(text)
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", *oracle.CFLAGS, "-I", os.path.dirname(SRC), "-o", str(lib), str(src), "-lm"],
                   check=True)
    return str(lib)


def _battery(lib):
    return subprocess.run([sys.executable, "-m", "tests._pin_battery", lib], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)


def test_unmodified_oracle_passes_battery(tmp_path):
    lib = _build(tmp_path, "orig", open(SRC).read())
    r = _battery(lib)
    assert r.returncode == 0, r.stdout + r.stderr


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation site for {name} not unique"
    lib = _build(tmp_path, name, text.replace(old, new))
    r = _battery(lib)
    assert r.returncode != 0, f"mutant {name} survived the pin battery"
