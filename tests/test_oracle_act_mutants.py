"""Pin strength of the actuation-model replay: plausible mistakes planted in
copies of ``oracle/tre_oracle_act.c`` (compiled on the CPU together with the
unmodified base oracle) must each fail at least one pin of act_pins.py."""
import os
import subprocess
import tempfile

import pytest

import oracle as O
import act_pins

HERE = os.path.dirname(O.__file__)
SRC_ACT = os.path.join(HERE, "tre_oracle_act.c")
SRC_BASE = os.path.join(HERE, "tre_oracle.c")

MUTANTS = {
    "complete_one_window_early": ("if (kind[m] != OA_NONE && until[m] < w) {",
                                  "if (kind[m] != OA_NONE && until[m] <= w) {"),
    "wake_ignores_delay": ("until[r] = w + wake_w;", "until[r] = w;"),
    "receiver_wakes_without_waiting_for_sleep": ("until[r] = w + sleep_w + wake_w;", "until[r] = w + wake_w;"),
    "donor_released_late": ("R[d] -= 1;  /* hidden from routing at once */", ""),
    "pool_counts_replicas": ("if (idle >= g[r]) {", "if (idle > 0) {"),
    "pool_not_charged_footprint": ("idle -= g[r];\n", "idle -= 1;\n"),
    "no_donor_feasibility": (" || idle < (int64_t)g[r] - g[m])", ")"),
    "shortfall_not_charged": ("if (short_by > 0) idle -= short_by;", ""),
    "excess_not_returned": ("ret[d] = short_by < 0 ? -short_by : 0;", "ret[d] = 0;"),
    "veto_ignored": (" || ((vetoed >> m) & 1u)", ""),
    "veto_wrong_tick": ("const uint64_t vetoed = veto ? veto[tick] : 0u;\n    tick += 1;",
                        "tick += 1;\n    const uint64_t vetoed = veto ? veto[tick] : 0u;"),
    "receiver_in_flight_again": ("if (ok[m] && kind[m] == OA_NONE && (r < 0 || Z[m] < Z[r])) r = m;",
                                 "if (ok[m] && (r < 0 || Z[m] < Z[r])) r = m;"),
    "donor_in_flight_again": ("if (!in_class || kind[m] != OA_NONE || m == r",
                              "if (!in_class || m == r"),
    "initial_budget_in_replicas": ("idle -= (int64_t)g[m] * R[m];", "idle -= R[m];"),
    "final_wakes_dropped": ("if (kind[m] != OA_NONE && until[m] < nW) {", "if (kind[m] != OA_NONE && until[m] < nW - 1) {"),
}


@pytest.fixture(scope="module")
def tmpdir():
    with tempfile.TemporaryDirectory() as d:
        yield d


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_act_mutant_is_caught(name, tmpdir):
    old, new = MUTANTS[name]
    text = open(SRC_ACT).read()
    assert text.count(old) == 1, f"mutant {name}: pattern not unique in the oracle"
    src = os.path.join(tmpdir, f"{name}.c")
    open(src, "w").write(text.replace(old, new))
    lib = os.path.join(tmpdir, f"lib{name}.so")
    subprocess.check_call(["gcc", *O.CFLAGS, "-o", lib, SRC_BASE, src, "-lm"])
    o = O.Oracle(lib)
    failed = []
    for pin in act_pins.ALL:
        try:
            pin(o)
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passes every pin"
