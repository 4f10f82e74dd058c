"""Pin strength of the closed-loop replay oracle: plausible mistakes planted
in copies of ``oracle/tre_oracle_loop.c`` (compiled on the CPU together with
the unmodified base oracle) must each fail at least one pin of
loop_pins.py."""
import os
import subprocess
import tempfile

import pytest

import oracle as O
import loop_pins

HERE = os.path.dirname(O.__file__)
SRC_LOOP = os.path.join(HERE, "tre_oracle_loop.c")
SRC_BASE = os.path.join(HERE, "tre_oracle.c")

MUTANTS = {
    "slot_that_frees_last": ("if (slot[m][k] < slot[m][best]) best = k;", "if (slot[m][k] > slot[m][best]) best = k;"),
    "move_acts_a_window_early": ("slot[r][(int64_t)R[r] * spr + q] = w_end;",
                                 "slot[r][(int64_t)R[r] * spr + q] = w_end - window_ms;"),
    "donor_releases_latest_free": ("if (slot[d][x] < slot[d][lo]) lo = x;", "if (slot[d][x] > slot[d][lo]) lo = x;"),
    "duration_floor_not_ceiling": ("return (tokens * (int64_t)us + 999) / 1000;", "return tokens * (int64_t)us / 1000;"),
    "replica_cap_ignored": ("if (ok[m] && !used[m] && R[m] < r_cap && (r < 0 || Z[m] < Z[r])) r = m;",
                            "if (ok[m] && !used[m] && (r < 0 || Z[m] < Z[r])) r = m;"),
    "idle_budget_ignored": ("      if (idle > 0) {\n        idle -= 1;", "      if (0) {\n        idle -= 1;"),
    "starts_past_the_window": ("        if (s >= w_end) break;", "        if (s >= duration_ms) break;"),
    "ttft_from_start": ("const int64_t ttft = t_first - arrival_ms[i], e2e = t - arrival_ms[i];",
                        "const int64_t ttft = t_first - s, e2e = t - arrival_ms[i];"),
    "donor_floor_ignored": ("R[m] <= prof[m].r_min || ", ""),
    "judged_past_the_end": ("if (t < duration_ms && t_first >= 0) {  /* judged */", "if (t_first >= 0) {"),
    "replicas_counted_after_the_moves": ("    for (int m = 0; m < M; ++m) r_windows[m] += R[m];\n", "\n"),
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
    subprocess.check_call(["gcc", *O.CFLAGS, "-o", lib, SRC_BASE, src, "-lm"])
    o = O.Oracle(lib)
    failed = []
    for pin in loop_pins.ALL:
        try:
            pin(o)
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passes every pin"
