"""Each plausible mistake planted in the oracle (on the CPU, in a throw-away
copy of its source) must fail at least one pin: the pins are strong enough to
catch a dropped term, a wrong sign, an off-by-one or a wrong tie-break."""
import os
import shutil
import subprocess
import tempfile

import pytest

import oracle
from tests import oracle_pins as pins

# (name, text in maps_oracle.c, replacement)
MUTANTS = [
    ("score_sign", "(int64_t)truth[i] - (int64_t)pred[i]", "(int64_t)pred[i] - (int64_t)truth[i]"),
    ("score_not_one_sided", "max64(0, (int64_t)truth[i] - (int64_t)pred[i])",
     "((int64_t)truth[i] - (int64_t)pred[i])"),
    ("rank_n_not_n_plus_1", "* (n + 1);", "* (n);"),
    ("rank_floor_not_ceil", "(num + 999999) / 1000000", "num / 1000000"),
    ("bucket_strict_edge", "if (edges[j] <= pred) b += 1;", "if (edges[j] < pred) b += 1;"),
    ("bound_minus_q", "(int64_t)pred[i] + qb", "(int64_t)pred[i] - qb"),
    ("bound_not_capped", "U_out[i] = (int32_t)min64((int64_t)pred[i] + qb, u_max);",
     "U_out[i] = (int32_t)((int64_t)pred[i] + qb);"),
    ("inf_quantile_gives_pred", "if (qb == ORACLE_Q_INF) U_out[i] = u_max;",
     "if (qb == ORACLE_Q_INF) U_out[i] = pred[i];"),
    ("missing_pred_gets_umax", "if (pred[i] < 0) { U_out[i] = -1; continue; }",
     "if (pred[i] < 0) { U_out[i] = u_max; continue; }"),
    ("occupancy_no_growth", "O[t] = held + t * active;", "O[t] = held;"),
    ("occupancy_leaves_early", "        O[t] = held + t * active;      /* every active request holds p+g+t */\n"
     "        active -= leave_cnt[t];        /* those whose last step is t leave */\n"
     "        held -= leave_tok[t];",
     "        active -= leave_cnt[t];\n        held -= leave_tok[t];\n        O[t] = held + t * active;"),
    ("remaining_plus_g", "return max64((int64_t)U - g, 0);", "return max64((int64_t)U - g + 1, 0);"),
    ("present_without_t", "max64(present[t - 1], O[t] + t)", "max64(present[t - 1], O[t])"),
    ("after_includes_u", "after[t] = max64(after[t + 1], O[t + 1]);", "after[t] = max64(after[t + 1], O[t]);"),
    ("peak_without_prompt", "max64((int64_t)a_p[a] + present[a_U[a]], after[a_U[a]])",
     "max64(present[a_U[a]], after[a_U[a]])"),
    ("feasible_strict", "if (policy == ORACLE_POLICY_MQ && slack >= 0) {",
     "if (policy == ORACLE_POLICY_MQ && slack > 0) {"),
    ("mq_ties_highest", "queue_len[d] < queue_len[feas_d[a]]", "queue_len[d] <= queue_len[feas_d[a]]"),
    ("fallback_ties_highest", "if (fb_d[a] < 0 || slack > fb_slack[a]) {",
     "if (fb_d[a] < 0 || slack >= fb_slack[a]) {"),
    ("fallback_min_slack", "if (fb_d[a] < 0 || slack > fb_slack[a]) {",
     "if (fb_d[a] < 0 || slack < fb_slack[a]) {"),
    ("rr_shifted", "choice[a] = (int32_t)((rr_offset + i) % D);", "choice[a] = (int32_t)((rr_offset + i + 1) % D);"),
    ("promotion_last", "keys[i].cls = promoted ? 0 : 1;", "keys[i].cls = promoted ? 1 : 0;"),
    ("promoted_by_bound", "keys[i].val = promoted ? i : Ui;", "keys[i].val = Ui;"),
    ("sjf_descending", "if (x->val != y->val) return x->val < y->val ? -1 : 1;",
     "if (x->val != y->val) return x->val > y->val ? -1 : 1;"),
    ("admission_no_growth", "G[t] += (int64_t)q_p[qlo + i] + t;", "G[t] += (int64_t)q_p[qlo + i];"),
    ("admission_strict", "if (peak > capacity[d]) break;", "if (peak >= capacity[d]) break;"),
    ("window_includes_seen", "if (pos[start[b] + mid] < seen[j]) lo = mid + 1;",
     "if (pos[start[b] + mid] <= seen[j]) lo = mid + 1;"),
    ("window_oldest_not_newest", "int64_t i = pos[start[b] + c - nw + t];", "int64_t i = pos[start[b] + t];"),
    ("window_rank_from_length", "int64_t k = oracle_conformal_rank(nw, alpha_ppm);",
     "int64_t k = oracle_conformal_rank(window, alpha_ppm);"),
    ("window_ignores_bucket", "int32_t b = oracle_bucket(apply_pred[j], edges, nb);", "int32_t b = 0;"),
    ("window_two_sided_score", "set[t] = max64(0, (int64_t)truth[i] - (int64_t)pred[i]);",
     "set[t] = (int64_t)truth[i] - (int64_t)pred[i];"),
    ("window_one_short", "int64_t nw = min64(c, window);", "int64_t nw = min64(c, window - 1);"),
    ("window_inf_gives_pred", "if (q == ORACLE_Q_INF) U_out[j] = u_max;", "if (q == ORACLE_Q_INF) U_out[j] = apply_pred[j];"),
    ("static_need_floor", "static int64_t ceil_div(int64_t x, int64_t s) { return (x + s - 1) / s; }",
     "static int64_t ceil_div(int64_t x, int64_t s) { return x / s; }"),
    ("static_feasible_strict", "if (need <= B[d] && (feas < 0 || Q[d] < Q[feas])) feas = d;",
     "if (need < B[d] && (feas < 0 || Q[d] < Q[feas])) feas = d;"),
    ("static_mq_ties_highest", "if (need <= B[d] && (feas < 0 || Q[d] < Q[feas])) feas = d;",
     "if (need <= B[d] && (feas < 0 || Q[d] <= Q[feas])) feas = d;"),
    ("static_fallback_ties_highest", "if (B[d] > B[most]) most = d;", "if (B[d] >= B[most]) most = d;"),
    ("static_no_reservation", "if (reserve) { B[best] -= need; Q[best] += 1; }", "if (reserve) { Q[best] += 1; }"),
    ("static_no_enqueue", "if (reserve) { B[best] -= need; Q[best] += 1; }", "if (reserve) { B[best] -= need; }"),
    ("static_rr_not_enqueued", "            if (reserve) Q[best] += 1;\n            continue;", "            continue;"),
    ("rsc_negative_reservation", "res += max64(demand - now, 0);", "res += demand - now;"),
    ("rsc_capacity_rounded_up", "b_free[d] = (int64_t)capacity[d] / S - held;",
     "b_free[d] = ceil_div(capacity[d], S) - held;"),
    ("blocks_gain_wrong_residue", "held += active_in[(S - t % S) % S];", "held += active_in[t % S];"),
    ("blocks_leave_one_late", "held -= (x + t + S - 1) / S;", "held -= (x + t + S) / S;"),
    ("blocks_start_floor", "held += (x + S - 1) / S;                 /* blocks at step 0 */",
     "held += x / S;                 /* blocks at step 0 */"),
    ("blocks_arrival_floor", "int64_t v = OB[t] + (rho + t + S - 1) / S;", "int64_t v = OB[t] + (rho + t) / S;"),
    ("blocks_capacity_rounded_up", "int64_t capB = (int64_t)capacity[d] / S;",
     "int64_t capB = ((int64_t)capacity[d] + S - 1) / S;"),
    ("blocks_prompt_residue_dropped", "int64_t P = a_p[a] / S, rho = a_p[a] % S;",
     "int64_t P = a_p[a] / S, rho = 0;"),
    ("bruteforce_extra_no_growth", "            if (t <= V[k]) occ += (int64_t)q[k] + t;",
     "            if (t <= V[k]) occ += (int64_t)q[k];"),
    ("bruteforce_resident_leaves_early", "if (t <= remaining(U[r], g[r])) occ += (int64_t)p[r] + g[r] + t;",
     "if (t < remaining(U[r], g[r])) occ += (int64_t)p[r] + g[r] + t;"),
    ("commit_no_growth", "for (int64_t t = 0; t <= a_U[a]; ++t) o[t] += (int64_t)a_p[a] + t;",
     "for (int64_t t = 0; t <= a_U[a]; ++t) o[t] += (int64_t)a_p[a];"),
    ("commit_not_applied", "o[t] += (int64_t)a_p[a] + t;", "o[t] += 0;"),
    ("commit_stale_prefix_max", "o[t] += (int64_t)a_p[a] + t;\n"
     "        for (int64_t t = 0; t <= T; ++t) pr[t] = (t == 0) ? o[0] : max64(pr[t - 1], o[t] + t);",
     "o[t] += (int64_t)a_p[a] + t;\n"),
    ("commit_queue_not_counted", "        choice[a] = best;\n        Q[best] += 1;", "        choice[a] = best;"),
    ("commit_rr_not_enqueued", "            flags[a] = 2;\n            Q[d] += 1;", "            flags[a] = 2;"),
    ("staged_in_flight_held", "res += U[r] < 0 ? ceil_div((int64_t)p[r], S) : ceil_div((int64_t)p[r] + U[r], S);",
     "held += U[r] < 0 ? ceil_div((int64_t)p[r], S) : ceil_div((int64_t)p[r] + U[r], S);"),
    ("staged_in_flight_prompt_only",
     "res += U[r] < 0 ? ceil_div((int64_t)p[r], S) : ceil_div((int64_t)p[r] + U[r], S);",
     "res += ceil_div((int64_t)p[r], S);"),
    ("sim_serves_newest", "int64_t i = rq[0];\n            for (int64_t k = 1; k < nready[d]; ++k) rq[k - 1] = rq[k];",
     "int64_t i = rq[nready[d] - 1];"),
    ("sim_run_to_completion", "else rq[nready[d]++] = i;",
     "else { for (int64_t k = nready[d]; k > 0; --k) rq[k] = rq[k - 1]; rq[0] = i; nready[d]++; }"),
    ("sim_fifo_bypass", "if (nfifo[d] == 0 && K[d] + DEMAND(i) <= C) {", "if (K[d] + DEMAND(i) <= C) {"),
    ("sim_pressure_strict", "if (K[d] * 1000000 >= (int64_t)theta_ppm * C) {",
     "if (K[d] * 1000000 > (int64_t)theta_ppm * C) {"),
    ("sim_finish_late", "finish_ms[release[d]] = t;", "finish_ms[release[d]] = t + 1;"),
    ("sim_no_reservation", "int64_t beff = C - K[k] - R[k];", "int64_t beff = C - K[k];"),
    ("sim_longest_queue", "(feas < 0 || nfifo[k] < nfifo[feas])", "(feas < 0 || nfifo[k] > nfifo[feas])"),
    ("sim_rr_shifted", "d = (int32_t)(i % N);", "d = (int32_t)((i + 1) % N);"),
    ("missing_bound_zero", "int64_t Ui = q_U[qlo + i] < 0 ? u_max : q_U[qlo + i];",
     "int64_t Ui = q_U[qlo + i] < 0 ? 0 : q_U[qlo + i];"),
]


def _build_mutant(tmp, name, old, new):
    with open(oracle.SOURCE) as f:
        src = f.read()
    assert old in src, f"mutation {name} does not apply"
    src = src.replace(old, new)
    path = os.path.join(tmp, f"{name}.c")
    with open(path, "w") as f:
        f.write(src)
    return oracle.build(path, os.path.join(tmp, f"lib{name}.so"), strict=False)


@pytest.fixture(scope="module")
def tmpdir_mutants():
    d = tempfile.mkdtemp(prefix="oracle_mutants_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_fails_a_pin(tmpdir_mutants, name, old, new):
    lib = oracle.load(_build_mutant(tmpdir_mutants, name, old, new))
    o = oracle.Oracle(lib)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(o)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
            break   # one failing pin is enough
    assert failed, f"planted mistake {name} passed every pin"


def test_unmutated_copy_passes(tmpdir_mutants):
    path = os.path.join(tmpdir_mutants, "liboriginal.so")
    o = oracle.Oracle(oracle.load(oracle.build(oracle.SOURCE, path)))
    for pin in pins.ALL_PINS:
        pin(o)
