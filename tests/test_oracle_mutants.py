"""Plant plausible mistakes in copies of the oracle source and check that the
pin suite rejects every one of them (no GPU).

Each mutant is a list of exact text replacements applied to
oracle/fate_oracle.c; the mutated copy is compiled into a temporary
directory, loaded, and run through every check in tests/pins.py.  A mutant
that passes every check would mean the pins cannot see that mistake.
"""

import os
import subprocess

import pytest

import pins
from oracle import oracle

MUTANTS = {
    "wait_not_clamped": [("return w > 0.0 ? w : 0.0;", "return w;")],
    "switch_even_if_resident": [("if (has_bit(s->res[d], m)) return 0.0;", "if (0) return 0.0;")],
    "transfer_beta_transposed": [("(double)in->beta[i * in->D + d] < bmin)\n                bmin = (double)in->beta[i * in->D + d];",
                                  "(double)in->beta[d * in->D + i] < bmin)\n                bmin = (double)in->beta[d * in->D + i];")],
    "transfer_first_holder": [("if (has_bit(hu, i) && (double)in->beta[i * in->D + d] < bmin)",
                               "if (has_bit(hu, i) && bmin == INFINITY)")],
    "transfer_child_size": [("tr += (double)in->sigma[s->base + u] * bmin;", "tr += (double)in->sigma[g] * bmin;")],
    "colo_sign": [("return c + t_sw + t_tr - t_co - t_pf - t_sm;", "return c + t_sw + t_tr + t_co - t_pf - t_sm;")],
    "colo_not_normalised": [("return (double)cnt / (double)np;", "return (double)cnt;")],
    "prefix_group_zero_counts": [("if (h == 0) return 0.0;", "if (0) return 0.0;")],
    "post_state_no_prefix": [("post.extra_hash[d] = in->hash[g];", "post.extra_hash[d] = 0;")],
    "post_state_no_holders": [("post.over_stage = v;", "post.over_stage = -1;")],
    "load_evicts_largest_id": [("for (int i = 0; i < in->M && total > in->cap[d]; ++i) {",
                                "for (int i = in->M - 1; i >= 0 && total > in->cap[d]; --i) {")],
    "load_never_evicts": [("res &= ~((uint64_t)1 << i);\n        total -= in->weight[i];",
                           "total -= in->weight[i];")],
    "depth_weight_off_by_one": [("pow(in->gamma, (double)sc.depth[w])", "pow(in->gamma, (double)(sc.depth[w] - 1))")],
    "horizon_one_level_too_deep": [("if (sc->depth[x] >= H) continue;", "if (sc->depth[x] > H) continue;")],
    "window_exec_not_split": [("double a_c = exec_c(in, mv, d) / k;", "double a_c = exec_c(in, mv, d);")],
    "window_transfer_not_split": [("transfer_cost(&cur, v, d) / k;", "transfer_cost(&cur, v, d);")],
    "window_switch_split": [("double a_s = in->lam_s * switch_cost(&cur, v, d);",
                             "double a_s = in->lam_s * switch_cost(&cur, v, d) / k;")],
    "window_wait_split": [("double a_q = in->lam_q * wait_cost(&cur, d);",
                           "double a_q = in->lam_q * wait_cost(&cur, d) / k;")],
    "gather_beta_transposed": [("in->beta[d * D + p]", "in->beta[p * D + d]")],
    "gather_max_over_target": [("gsum = INFINITY;", "gsum = -INFINITY;"), ("if (s < gsum) gsum = s;", "if (s > gsum) gsum = s;")],
    "feasible_ignores_capacity": [("return has_bit(in->elig[g], d) && fits(in, in->model[g], d);",
                                   "return has_bit(in->elig[g], d);")],
    "feasible_ignores_eligibility": [("return has_bit(in->elig[g], d) && fits(in, in->model[g], d);",
                                      "return fits(in, in->model[g], d);")],
    "frontier_includes_running": [("if (in->status[g] != ST_PENDING) return 0;",
                                   "if (in->status[g] == ST_COMPLETED) return 0;")],
    "descendant_max_device": [("if (val < vbest) { vbest = val; vmag = m_; }",
                               "if (vbest == INFINITY || val > vbest) { vbest = val; vmag = m_; }")],
    "prefix_sign": [("return c + t_sw + t_tr - t_co - t_pf - t_sm;", "return c + t_sw + t_tr - t_co + t_pf - t_sm;")],
    # the magnitude A that parity tolerances divide by
    "mag_gamma_dropped": [("A += gw_pow * vmag;", "A += vmag;")],
    "mag_all_horizon_devices": [("if (val < vbest) { vbest = val; vmag = m_; }",
                                 "vmag += m_;\n                    if (val < vbest) vbest = val;")],
    "mag_all_shard_devices": [("best_mag = fabs(a_q) + fabs(a_c)", "best_mag += fabs(a_q) + fabs(a_c)")],
    "mag_gather_twice": [("double A = best_mag + fabs(in->lam_tr * gsum);",
                          "double A = best_mag + 2.0 * fabs(in->lam_tr * gsum);")],
    "mag_horizon_max_device": [("if (val < vbest) { vbest = val; vmag = m_; }",
                                "if (val < vbest) vbest = val;\n                    if (m_ > vmag) vmag = m_;")],
    "mag_signed_benefit": [("if (mag) *mag = fabs(c) + fabs(t_sw) + fabs(t_tr) + fabs(t_co) + fabs(t_pf) + fabs(t_sm);",
                            "if (mag) *mag = fabs(c) + fabs(t_sw) + fabs(t_tr) - fabs(t_co) - fabs(t_pf) + fabs(t_sm);")],
    # commit-and-advance
    "commit_start_ignores_now": [("double start = tau_out[bd] > (double)in->t_now[b] ? tau_out[bd] : (double)in->t_now[b];",
                                  "double start = tau_out[bd];")],
    "commit_switch_always": [("double sw = has_bit(res_out[bd], m) ? 0.0 : (double)in->switch_s[m * D + d];",
                              "double sw = (double)in->switch_s[m * D + d];")],
    "commit_exec_not_split": [("tau_out[bd] = start + exec_c(in, m, d) / (double)k + sw;",
                               "tau_out[bd] = start + exec_c(in, m, d) + sw;")],
    "commit_full_ring_overwrites_newest": [("for (int q = 0; q + 1 < K; ++q) slots[q] = slots[q + 1];\n", "")],
    "commit_holders_last_device": [("held |= (uint64_t)1 << d;", "held = (uint64_t)1 << d;")],
    "commit_no_load": [("res_out[bd] = load_model(in, res_out[bd], m, d);", "res_out[bd] = res_out[bd];")],
    "commit_ignores_feasibility": [("if (!ok) { ++rejected; continue; }", "if (0) { ++rejected; continue; }")],
    "commit_not_completed": [("status_out[g] = ST_COMPLETED;", "status_out[g] = status_out[g];")],
    "commit_ignores_inputs": [("                    if (arr > start) start = arr;\n", "")],
    "commit_input_not_split": [("arr = fin_io[u] + (double)in->sigma[u] * bmin / (double)k;",
                                "arr = fin_io[u] + (double)in->sigma[u] * bmin;")],
    "commit_local_input_transferred": [("                    if (!has_bit(holders_out[u], d)) {\n                        double bmin",
                                        "                    if (1) {\n                        double bmin")],
    "commit_finish_first_shard": [("if (tau_out[bd] > fin) fin = tau_out[bd];", "if (fin == -INFINITY) fin = tau_out[bd];")],
    # scoring variants
    "same_model_when_absent": [("return has_bit(s->res[d], s->in->model[s->base + x]) ? 1.0 : 0.0;",
                                "return has_bit(s->res[d], s->in->model[s->base + x]) ? 0.0 : 1.0;")],
    "same_model_not_in_horizon": [("double t_sm = in->lam_m * same_model(s, x, d);", "double t_sm = 0.0;")],
    "same_model_not_immediate": [("double a_sm = in->lam_m * same_model(&cur, v, d);", "double a_sm = 0.0;")],
    "same_model_in_current_state": [("double t_sm = in->lam_m * same_model(s, x, d);",
                                     "double t_sm = in->lam_m * (has_bit(s->in->resident[(int64_t)s->b * s->in->D + d], "
                                     "s->in->model[s->base + x]) ? 1.0 : 0.0);")],
    "topo_level_min_parent": [("if (l > sc.level[x]) sc.level[x] = l;",
                               "if (sc.level[x] == 0 || l < sc.level[x]) sc.level[x] = l;")],
    "topo_depth_is_hops": [("sc->depth[c] = dl;", "sc->depth[c] = sc->depth[x] + 1;")],
    "mean_over_all_levels": [("if (in->mean_levels) gw_pow /= (double)sc.nlev[sc.depth[w]];",
                              "if (in->mean_levels) gw_pow /= (double)count;")],
    "no_windows_ignored": [("if (!ok || (k > 1 && in->no_windows))", "if (!ok)")],
    # frontier planning wave
    "plan_ties_to_later": [("if (best_f < 0 || v > best_v)", "if (best_f < 0 || v >= best_v)")],
    "plan_ignores_devices": [("if (m & used) continue;", "if (0) continue;")],
    "plan_window_one_device": [("for (int d = i0; d < i0 + w; ++d) m |= (uint64_t)1 << d;", "m = (uint64_t)1 << i0;")],
    "plan_takes_inf": [("if (j < 0 || j >= n_cand[f] || v == -INFINITY) continue;",
                        "if (j < 0 || j >= n_cand[f]) continue;")],
    "plan_past_candidates": [("if (j < 0 || j >= n_cand[f] || v == -INFINITY) continue;",
                              "if (j < 0 || v == -INFINITY) continue;")],
    "plan_stage_twice": [("if (sel_out[f] >= 0) continue;", "if (0) continue;")],
}


def _build_mutant(name, tmp_path):
    src = open(oracle.SRC).read()
    for old, new in MUTANTS[name]:
        assert src.count(old) == 1, (name, old)
        src = src.replace(old, new)
    cpath = os.path.join(tmp_path, name + ".c")
    with open(cpath, "w") as fh:
        fh.write(src)
    so = os.path.join(tmp_path, "lib" + name + ".so")
    subprocess.run(["gcc", "-O1", "-std=c11", "-fopenmp", "-shared", "-fPIC", cpath, "-o", so, "-lm"], check=True)
    return oracle.load(so)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name, tmp_path):
    lib = _build_mutant(name, str(tmp_path))
    caught = []
    for check_name, check in pins.ALL_CHECKS:
        try:
            check(lib)
        except AssertionError:
            caught.append(check_name)
            break
    assert caught, "no pin rejects the planted mistake '%s'" % name
