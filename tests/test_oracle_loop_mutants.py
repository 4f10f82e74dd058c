"""Pin strength of the closed-loop replay oracle: plausible mistakes planted
in copies of ``oracle/tre_oracle_loop.c`` (compiled on the CPU together with
the unmodified base and actuation oracles) must each fail at least one pin
of loop_pins.py."""
import os
import subprocess
import tempfile

import pytest

import oracle as O
import loop_pins

HERE = os.path.dirname(O.__file__)
SRC_LOOP = os.path.join(HERE, "tre_oracle_loop.c")
SRC_BASE = os.path.join(HERE, "tre_oracle.c")
SRC_ACT = os.path.join(HERE, "tre_oracle_act.c")  # the actuation replay, which pins the closed loop's moves

MUTANTS = {
    "slot_that_frees_last": ("if (slot[m][k] < slot[m][best]) best = k;", "if (slot[m][k] > slot[m][best]) best = k;"),
    "move_acts_a_window_early": ("slot[m][(int64_t)R[m] * spr + q] = w * window_ms;",
                                 "slot[m][(int64_t)R[m] * spr + q] = (w - 1) * window_ms;"),
    "donor_releases_latest_free": ("if (slot[d][x] < slot[d][lo]) lo = x;", "if (slot[d][x] > slot[d][lo]) lo = x;"),
    "duration_floor_not_ceiling": ("return (tokens * (int64_t)us + 999) / 1000;", "return tokens * (int64_t)us / 1000;"),
    "replica_cap_ignored": ("if (ok[m] && kind[m] == OL_NONE && R[m] < r_cap && (r < 0 || Z[m] < Z[r])) r = m;",
                            "if (ok[m] && kind[m] == OL_NONE && (r < 0 || Z[m] < Z[r])) r = m;"),
    "idle_budget_ignored": ("      if (idle >= g[r]) {\n        idle -= g[r];", "      if (0) {\n        idle -= g[r];"),
    "starts_past_the_window": ("        if (s >= w_end) break;", "        if (s >= duration_ms) break;"),
    "ttft_from_start": ("const int64_t ttft = t_first - arrival_ms[i], e2e = t - arrival_ms[i];",
                        "const int64_t ttft = t_first - s, e2e = t - arrival_ms[i];"),
    "donor_floor_ignored": ("R[m] <= prof[m].r_min || ", ""),
    "judged_past_the_end": ("if (t < duration_ms && t_first >= 0) {  /* judged */", "if (t_first >= 0) {"),
    "replicas_counted_after_the_moves": ("    for (int m = 0; m < M; ++m) r_windows[m] += R[m];\n", "\n"),
    # the actuation model
    "transition_completes_a_window_early": ("if (kind[m] != OL_NONE && until[m] < w) {",
                                            "if (kind[m] != OL_NONE && until[m] <= w) {"),
    "footprint_ignored_on_the_pool_path": ("      if (idle >= g[r]) {\n        idle -= g[r];",
                                           "      if (idle >= 1) {\n        idle -= 1;"),
    "receiver_wakes_before_the_sleep": ("until[r] = w + sleep_w + wake_w;", "until[r] = w + wake_w;"),
    "vetoes_ignored": ("((vetoed >> m) & 1u) || ", ""),
    "waking_model_receives_again": ("if (ok[m] && kind[m] == OL_NONE && R[m] < r_cap",
                                    "if (ok[m] && kind[m] != OL_SLEEP && R[m] < r_cap"),
    "excess_not_returned": ("ret[d] = short_by < 0 ? -short_by : 0;", "ret[d] = 0;"),
    "shortfall_not_charged": ("if (short_by > 0) idle -= short_by;", ""),
    "donor_feasibility_unchecked": (" ||\n                ((vetoed >> m) & 1u) || idle < (int64_t)g[r] - g[m])",
                                    " ||\n                ((vetoed >> m) & 1u))"),
    "veto_read_a_tick_late": ("const uint64_t vetoed = veto ? veto[tick] : 0u;",
                              "const uint64_t vetoed = veto ? veto[tick > 0 ? tick - 1 : 0] : 0u;"),
}


@pytest.fixture(scope="module")
def tmpdir():
    with tempfile.TemporaryDirectory() as d:
        yield d


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_loop_mutant_is_caught(name, tmpdir):
    old, new = MUTANTS[name]
    text = open(SRC_LOOP).read()
    assert text.count(old) == 1, f"mutant {name}: pattern not unique in the oracle"
    src = os.path.join(tmpdir, f"{name}.c")
    open(src, "w").write(text.replace(old, new))
    lib = os.path.join(tmpdir, f"lib{name}.so")
    subprocess.check_call(["gcc", *O.CFLAGS, "-o", lib, SRC_BASE, SRC_ACT, src, "-lm"])
    o = O.Oracle(lib)
    failed = []
    # the quick hand-derived pins first: a mutant stops at its first failure
    quick = [p for p in loop_pins.ALL if "hand" in p.__name__ or "earliest" in p.__name__ or "bad_arg" in p.__name__]
    for pin in quick + [p for p in loop_pins.ALL if p not in quick]:
        try:
            pin(o)
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
            break  # one failing pin is enough
    assert failed, f"mutant {name} passes every pin"
