"""The pins are strong enough: plant one plausible mistake at a time in a copy
of the oracle's C source, build it, and require that at least one pin fails.

Planted mistakes stay on the CPU, in temporary copies of the oracle.
"""
import os
import subprocess
import sys

import pytest

import oracle
from oracle_pins import ALL_PINS

_SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

# (name, text in oracle.c, replacement)
MUTANTS = [
    ("spec_residual_unclipped", "w[i] = r > 0.0 ? r : 0.0;", "w[i] = r;"),
    ("spec_accept_inverted", "if (!(u_acc[(size_t)b * max_k + m] * q < p)) break;",
     "if (!(u_acc[(size_t)b * max_k + m] * p < q)) break;"),
    ("spec_accept_ratio_capped_low", "if (!(u_acc[(size_t)b * max_k + m] * q < p)) break;",
     "if (!(u_acc[(size_t)b * max_k + m] < 0.5 * p / q)) break;"),
    ("spec_bonus_from_last_draft_row",
     "const float *t = tlogits + ((size_t)b * (max_k + 1) + m) * row_stride;\n        double mt, zt;",
     "const float *t = tlogits + ((size_t)b * (max_k + 1) + (m == k && m > 0 ? m - 1 : m)) * row_stride;\n        double mt, zt;"),
    ("spec_residual_from_target_only", "const double r = row_prob(t, i, tau, mt, zt) - row_prob(d, i, tau, md, zd);",
     "const double r = row_prob(t, i, tau, mt, zt);"),
    ("spec_draft_tau_ignored", "const double q = row_prob(d, x, tau, md, zd);",
     "const double q = row_prob(d, x, 1.0, md, zd);"),
    ("spec_inversion_ge", "if (run > target) return i;", "if (run >= target) return i;"),
    ("drop_softmax_scale", "x[i] = sm_scale * dot;", "x[i] = dot;"),
    ("gqa_head_interleaved", "const int h = c * g + hh;", "const int h = hh * n_kv_heads + c;"),
    ("causal_off_by_one", "const int p = T - nq + j;", "const int p = T - nq + j - 1;"),
    ("causal_dropped", "const int p = T - nq + j;", "const int p = T - 1;"),
    ("window_off_by_one", "(j >= nq - w)", "(j > nq - w)"),
    ("scores_unnormalized", "if (in_window) S[i] += P;", "if (in_window) S[i] += x[i];"),
    ("scores_first_rows", "(j >= nq - w)", "(j < w)"),
    ("max_not_subtracted_twice", "x[i] = exp(x[i] - m);\n                    L += x[i];",
     "x[i] = exp(x[i] - m);\n                    L += 1.0;"),
    ("tie_to_higher_position", "return (a->i > b->i) - (a->i < b->i);",
     "return (a->i < b->i) - (a->i > b->i);"),
    ("ascending_scores", "if (a->s > b->s) return -1;\n    if (a->s < b->s) return 1;",
     "if (a->s < b->s) return -1;\n    if (a->s > b->s) return 1;"),
    ("recent_off_by_one", "const int r_start = (T - k_recent) > s_end ? (T - k_recent) : s_end;\n"
     "        const int n_mid", "const int r_start = (T - k_recent + 1) > s_end ? "
     "(T - k_recent + 1) : s_end;\n        const int n_mid"),
    ("sink_not_kept", "for (int i = 0; i < s_end; ++i) keep[i] = 1;", ""),
    ("kmid_ignores_sink", "const int k_mid = budget - k_sink - k_recent;\n\n#pragma omp parallel for"
     " schedule(dynamic, 1)\n    for (int u = 0; u < batch * n_kv_heads; ++u) {",
     "const int k_mid = budget - k_recent;\n\n#pragma omp parallel for schedule(dynamic, 1)\n"
     "    for (int u = 0; u < batch * n_kv_heads; ++u) {"),
    ("draft_head_modulo", "const int b = bh / n_q_heads, h = bh % n_q_heads, c = h / g;",
     "const int b = bh / n_q_heads, h = bh % n_q_heads, c = h % n_kv_heads;"),
    ("draft_drops_last_index", "for (int t = 0; t < n; ++t) {\n            double dot",
     "for (int t = 0; t < n - 1; ++t) {\n            double dot"),
    ("step_window_not_slid", "const int w0 = (cur - k_recent) > r_T ? (cur - k_recent) : r_T;",
     "const int w0 = r_T;"),
    ("step_fixed_part_inclusive", "if (I[t] < r_T) S[m_S++] = I[t];", "if (I[t] <= r_T) S[m_S++] = I[t];"),
    ("step_window_misses_newest", "for (int t = w0; t < cur; ++t) S[m_S++] = t;",
     "for (int t = w0; t < cur - 1; ++t) S[m_S++] = t;"),
    ("step_fixed_part_from_cur", "const int r_T = (T - k_recent) > s_end ? (T - k_recent) : s_end;",
     "const int r_T = (cur - k_recent) > s_end ? (cur - k_recent) : s_end;"),
    ("step_heads_use_group_set", "const int32_t *I = per_head ? idx + ((size_t)b * n_q_heads + h) * budget",
     "const int32_t *I = per_head ? idx + ((size_t)b * n_q_heads + c * g) * budget"),
    ("step_heads_ignore_own_set", "const int32_t *I = per_head ? idx",
     "const int32_t *I = 0 ? idx"),
    ("entropy_log2", "const double lp = x[i] - m - log(Z);      /* ln p_i */",
     "const double lp = (x[i] - m - log(Z)) / log(2.0);"),
    ("entropy_unnormalized", "const double lp = x[i] - m - log(Z);      /* ln p_i */",
     "const double lp = x[i] - m;"),
    ("argmax_ties_to_last", "if (x[i] > x[a]) a = i;", "if (x[i] >= x[a]) a = i;"),
    ("accept_one_past_mismatch", "while (m < k_len[b] && db[m] == tb[m]) ++m;",
     "while (m < k_len[b] && db[m] == tb[m]) ++m;\n            if (m < k_len[b]) ++m;"),
    ("next_token_from_row_after", "next_token[b] = tb[m];", "next_token[b] = tb[m < k_len[b] ? m + 1 : m];"),
    ("head_scores_kv_head_modulo", "const int b = bh / n_q_heads, h = bh % n_q_heads, c = h / g;\n        const int T = ctx_len[b], nq = q_len[b];",
     "const int b = bh / n_q_heads, h = bh % n_q_heads, c = h % n_kv_heads;\n        const int T = ctx_len[b], nq = q_len[b];"),
    ("head_scores_all_rows", "for (int j = nq - w; j < nq; ++j) {", "for (int j = 0; j < nq; ++j) {"),
    ("draft_heads_shared_set", "const int32_t *I = idx + ((size_t)b * n_q_heads + h) * budget;",
     "const int32_t *I = idx + ((size_t)b * n_q_heads + c * g) * budget;"),
    ("ema_weights_swapped", "return beta * prev + (1.0 - beta) * observed;",
     "return beta * observed + (1.0 - beta) * prev;"),
    ("observe_no_first_init", "if (state[2 + cls] != 0.0)", "if (1)"),
    ("observe_empty_label_updated", "if (hi == lo) continue;                 /* no token carries this label */", ""),
    ("observe_split_off_by_one", "const int lo = cls == 0 ? 0 : n_accepted;",
     "const int lo = cls == 0 ? 0 : n_accepted + 1;"),
    ("observe_mean_over_all_drafts", "for (int i = lo; i < hi; ++i) sum += H[i];",
     "for (int i = 0; i < n_drafted; ++i) sum += H[i];"),
    ("observe_seen_flag_not_set", "        state[2 + cls] = 1.0;\n", ""),
    ("accept_prob_inverted", "return ea / (ea + er);", "return er / (ea + er);"),
    ("expected_drops_last_term", "for (int m = 1; m <= k; ++m) {", "for (int m = 1; m < k; ++m) {"),
    ("expected_sum_not_product", "for (int i = 0; i < m; ++i) prod *= p[i];",
     "for (int i = 0; i < m; ++i) prod = p[i];"),
    ("objective_no_correction_token", "return (1.0 + oracle_expected_accepted(p, k))",
     "return (oracle_expected_accepted(p, k))"),
    ("argmax_ties_to_larger", "(val == best_val && k < best)", "(val == best_val && k > best)"),
    ("argmax_allows_unknown_k", "if (k < 0 || k > n) continue;", "if (k < 0) continue;"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(name, old, new, tmp_path):
    src = open(_SRC).read()
    assert src.count(old) >= 1, f"mutation anchor for {name} not found in oracle.c"
    mutated = src.replace(old, new, 1)
    csrc = tmp_path / "oracle_mutant.c"
    csrc.write_text(mutated)
    so = tmp_path / "liboracle_mutant.so"
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11", str(csrc),
                    "-o", str(so), "-lm"], check=True)
    # The pins run in a child process: a planted out-of-bounds write may abort it,
    # which also counts as the mistake being caught.
    code = (
        "import sys, oracle\n"
        "from oracle_pins import ALL_PINS\n"
        f"lib = oracle.load({str(so)!r})\n"
        "caught = []\n"
        "for pin in ALL_PINS:\n"
        "    try:\n"
        "        pin(lib)\n"
        "    except (AssertionError, ValueError, IndexError):\n"
        "        caught.append(pin.__name__)\n"
        "print('CAUGHT', ' '.join(caught))\n"
        "sys.exit(0 if caught else 3)\n")
    env = dict(os.environ)
    here = os.path.dirname(os.path.abspath(__file__))
    env["PYTHONPATH"] = os.pathsep.join([os.path.dirname(here), here, env.get("PYTHONPATH", "")])
    env["OMP_NUM_THREADS"] = "2"
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode != 3, f"no pin catches the planted mistake {name}:\n{r.stdout}{r.stderr}"
    if r.returncode == 0:
        assert "CAUGHT" in r.stdout
