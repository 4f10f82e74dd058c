"""Pin strength: plausible mistakes planted in copies of the oracle.

Each mutant is a text edit of ``oracle/tre_oracle.c`` (a dropped term, a
wrong sign or index, a swapped operand, a flipped comparison).  The edited
copy is compiled on the CPU into a temporary library and every pin of
``pins.py`` is run against it; at least one pin must fail.  The real oracle
is never modified.
"""
import os
import tempfile

import pytest

import oracle as O
import pins

SRC = os.path.join(os.path.dirname(O.__file__), "tre_oracle.c")

MUTANTS = {
    # Eq. (1) numerator / denominator
    "drop_prefill_weight": ("double num = w_p * (double)P;", "double num = (double)P;"),
    "prefill_weight_on_decode": ("num = num + (double)D;", "num = num + w_p * (double)D;"),
    "drop_waiting_weight": ("double q = w_q * (double)W_int;", "double q = (double)W_int;"),
    "drop_active_term": ("double den = (double)A_int + q;", "double den = q;"),
    "drop_waiting_term": ("double den = (double)A_int + q;", "double den = (double)A_int;"),
    "no_floor": ("if (den < (double)window_ms) den = (double)window_ms;", ""),
    "floor_wrong_unit": ("if (den < (double)window_ms) den = (double)window_ms;",
                         "if (den < 1.0) den = 1.0;"),
    "rate_per_ms": ("num = num * 1000.0;", ""),
    # smoothing
    "swap_alpha_weights": ("double t1 = alpha * raw;", "double t1 = (1.0 - alpha) * raw;"),
    "prev_weight_alpha": ("double t2 = (1.0 - alpha) * s_prev;", "double t2 = alpha * s_prev;"),
    "init_to_zero": ("else { s = raw; init = 1; }", "else { s = oracle_smooth(prof[m].alpha, raw, 0.0); init = 1; }"),
    "no_idle_hold": ("const int idle = P[c] == 0 && D[c] == 0 && A_int[c] == 0 && W_int[c] == 0;",
                     "const int idle = 0;"),
    # window observations
    "arrive_not_waiting": ("case OR_ARRIVE: W[m] += 1; break;", "case OR_ARRIVE: break;"),
    "admit_keeps_waiting": ("if (admit) { W[m] -= 1; A[m] += 1; }", "if (admit) { A[m] += 1; }"),
    "finish_not_leaving": ("case OR_FINISH: A[m] -= 1; break;", "case OR_FINISH: break;"),
    "prefill_into_decode": ("P[w * M + m] += tokens[i];", "D[w * M + m] += tokens[i];"),
    "integral_off_by_one": ("integ[w * M + m] += count * (seg_end - from);",
                            "integ[w * M + m] += count * (seg_end - from + 1);"),
    "integral_wrong_window": ("int64_t w = from / window_ms;", "int64_t w = (from + 1) / window_ms;"),
    "no_tail_integral": ("integrate(A_int, M, m, window_ms, A[m], t_last[m], duration_ms);", ""),
    # normalisation and regions
    "theta_divided_by_scale": ("theta_eff[m] = prof[m].theta * sc->theta_scale;",
                               "theta_eff[m] = prof[m].theta / sc->theta_scale;"),
    "ignore_tau_override": ("tau_c[m] = sc->tau_crit_override >= 0.0 ? sc->tau_crit_override : prof[m].tau_crit;",
                            "tau_c[m] = prof[m].tau_crit;"),
    "crit_non_strict": ("crit[m] = Z[m] < tau_c[m];", "crit[m] = Z[m] <= tau_c[m];"),
    "surplus_non_strict": ("surplus[m] = Z[m] > prof[m].tau_surplus;", "surplus[m] = Z[m] >= prof[m].tau_surplus;"),
    "idle_reads_S": ("Z[m] = ((f & OR_IDLE) || !(f & OR_INIT)) ? INFINITY : S[w * M + m] / theta_eff[m];",
                     "Z[m] = !(f & OR_INIT) ? INFINITY : S[w * M + m] / theta_eff[m];"),
    # dual-speed control
    "no_defer": ("if (!fast) continue;", ""),
    "rescue_any_tick": ("const int fast = t_end % fast_ms == 0;", "const int fast = 1;"),
    "rebalance_any_receiver": ("for (int m = 0; m < M; ++m) ok[m] = Z[m] < 1.0;",
                               "for (int m = 0; m < M; ++m) ok[m] = 1;"),
    "rebalance_at_fast": ("} else if (slow) {", "} else if (slow || fast) {"),
    "rescue_all_below_one": ("for (int m = 0; m < M; ++m) ok[m] = crit[m];",
                             "for (int m = 0; m < M; ++m) ok[m] = Z[m] < 1.0;"),
    # receiver / donor selection
    "receiver_argmax": ("if (ok[m] && !used[m] && (r < 0 || Z[m] < Z[r])) r = m;",
                        "if (ok[m] && !used[m] && (r < 0 || Z[m] > Z[r])) r = m;"),
    "receiver_tie_highest": ("if (ok[m] && !used[m] && (r < 0 || Z[m] < Z[r])) r = m;",
                             "if (ok[m] && !used[m] && (r < 0 || Z[m] <= Z[r])) r = m;"),
    "receiver_reuse": ("if (ok[m] && !used[m] && (r < 0 || Z[m] < Z[r])) r = m;",
                       "if (ok[m] && (r < 0 || Z[m] < Z[r])) r = m;"),
    "donor_tie_highest": ("if (best < 0 || Z[m] > Z[best]) best = m;", "if (best < 0 || Z[m] >= Z[best]) best = m;"),
    "donor_argmin": ("if (best < 0 || Z[m] > Z[best]) best = m;", "if (best < 0 || Z[m] < Z[best]) best = m;"),
    "nominal_first": ("const int in_class = pass == 0 ? surplus[m] : nominal;",
                      "const int in_class = pass == 0 ? nominal : surplus[m];"),
    "no_class_order": ("const int in_class = pass == 0 ? surplus[m] : nominal;",
                       "const int in_class = surplus[m] || nominal;"),
    "floor_non_strict": ("R[m] <= prof[m].r_min", "R[m] < prof[m].r_min"),
    "no_healthier_check": (" || !(Z[m] > Z[r]))", ")"),
    "donor_reuse": ("if (!in_class || used[m] || m == r", "if (!in_class || m == r"),
    "pool_ignored": ("if (pool > 0) {", "if (0) {"),
    "receiver_not_incremented": ("      R[r] += 1;\n      used[r] = 1;", "      used[r] = 1;"),
    "r_windows_after_tick": ("for (int m = 0; m < M; ++m) r_windows[m] += R[m];   /* replicas serving window w */",
                             "for (int m = 0; m < M; ++m) if (w > 0) r_windows[m] += R[m];"),
    "window_index_shift": ("moves[nm].window = (uint32_t)w;", "moves[nm].window = (uint32_t)(w + 1);"),
    # counts never negative (readings of Eq. (1)'s definition)
    "state_unchecked": ("if (A[k] < 0 || W[k] < 0) return -5;", ";"),
    "state_active_only": ("if (A[k] < 0 || W[k] < 0)", "if (A[k] < 0)"),
    "state_after_every_row": ("if (i == n_events - 1 || ts[i + 1] != t)", "if (1)"),
    "state_at_end_only": ("if (i == n_events - 1 || ts[i + 1] != t)", "if (i == n_events - 1)"),
    "state_own_model_only": ("for (int k = 0; k < M; ++k)\n        if (A[k] < 0", "for (int k = m; k <= m; ++k)\n        if (A[k] < 0"),
    "admits_unchecked": ("if (ids_scratch[i] == ids_scratch[i - 1]) {", "if (0) {"),
    "lifecycle_unchecked": ("    if (arrivals > 1 || finishes > 1 || (finishes == 1 && last_ad_ts > fin_ts)) {",
                            "    if (0) {"),
    "lifecycle_same_instant": ("(finishes == 1 && last_ad_ts > fin_ts)", "(finishes == 1 && last_ad_ts >= fin_ts)"),
    "lifecycle_arrivals_free": ("if (arrivals > 1 || finishes > 1", "if (finishes > 1"),
    "lifecycle_finishes_free": ("if (arrivals > 1 || finishes > 1 ||", "if (arrivals > 1 ||"),
    "lifecycle_decode_free": ("        if (kind == OR_ARRIVE) ++arrivals;\n        if (ts[row] > last_ad_ts) last_ad_ts = ts[row];",
                              "        if (kind == OR_ARRIVE) ++arrivals;\n        if (kind == OR_ARRIVE && ts[row] > last_ad_ts) last_ad_ts = ts[row];"),
    "lifecycle_prefill_counted": ("    if (kind == OR_ARRIVE || kind == OR_DECODE || kind == OR_FINISH)\n      keys_scratch",
                                  "    if (1)\n      keys_scratch"),
    "admits_any_prefill": ("if (type[i] == (OR_PREFILL | OR_ADMIT)) ids_scratch[n++] = req[i];",
                           "if ((type[i] & 3) == OR_PREFILL) ids_scratch[n++] = req[i];"),
    "no_move_limit": ("for (uint32_t k = 0; k < sc->max_moves; ++k) {", "for (uint32_t k = 0; k < sc->max_moves + 1; ++k) {"),
}


def _compile(name, old, new, tmpdir):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutant {name}: pattern not found"
    mutated = src.replace(old, new, 1)
    assert mutated != src
    path = os.path.join(tmpdir, f"{name}.c")
    with open(path, "w") as f:
        f.write(mutated)
    return O.build(force=True, src=path, out=os.path.join(tmpdir, f"lib{name}.so"))


@pytest.fixture(scope="module")
def tmpdir():
    with tempfile.TemporaryDirectory() as d:
        yield d


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmpdir):
    old, new = MUTANTS[name]
    lib = _compile(name, old, new, tmpdir)
    o = O.Oracle(lib)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(o)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} survived every pin"
