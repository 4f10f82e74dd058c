"""Pin strength of the calibration-sweep oracle: plausible mistakes planted
in copies of ``oracle/tre_oracle_calib.c`` (compiled on the CPU together
with the unmodified base oracle) must each fail at least one pin of
calib_pins.py."""
import os
import subprocess
import tempfile

import pytest

import oracle as O
import calib_pins

HERE = os.path.dirname(O.__file__)
SRC_CALIB = os.path.join(HERE, "tre_oracle_calib.c")
SRC_BASE = os.path.join(HERE, "tre_oracle.c")

MUTANTS = {
    "last_decode_as_first": ("if (f[r] == OC_NONE) f[r] = (uint32_t)i;", "f[r] = (uint32_t)i;"),
    "tpot_over_all_decode_tokens": ("const uint64_t after_first = d[r] - tokens[f[r]];",
                                    "const uint64_t after_first = d[r];"),
    "decode_events_not_tokens": ("d[r] += tokens[i];", "d[r] += 1;"),
    "window_of_finish": ("const int64_t w = ts[a[r]] / window_ms;", "const int64_t w = ts[e[r]] / window_ms;"),
    "strict_ttft_bound": ("(double)q.ttft_ms <= slo[m].ttft_ms", "(double)q.ttft_ms < slo[m].ttft_ms"),
    "e2e_bound_ignored": (" && (double)q.e2e_ms <= slo[m].e2e_ms;", ";"),
    "tpot_bound_ignored": ("good = good && q.tpot_ms <= slo[m].tpot_ms;", ""),
    "bad_ids_not_counted": ("      ++bad;\n", "\n"),
    "strict_window_health": (">= slo[m].attain_q * (double)j;", "> slo[m].attain_q * (double)j;"),
    "strict_reliability": ("(double)H >= slo[m].reliability * (double)N", "(double)H > slo[m].reliability * (double)N"),
    "ties_split": ("while (j < k && c[j].s == c[i].s) {", "while (j < k && j == i) {"),
    "largest_qualifying_threshold": ("if ((double)H >= slo[m].reliability * (double)N) {",
                                     "if (isinf(best.theta) && (double)H >= slo[m].reliability * (double)N) {"),
    "idle_windows_are_candidates": ("if (j == 0 || !(fl & OC_INIT) || (fl & OC_IDLE)) continue;",
                                    "if (j == 0 || !(fl & OC_INIT)) continue;"),
    "empty_windows_are_candidates": ("if (j == 0 || !(fl & OC_INIT) || (fl & OC_IDLE)) continue;",
                                     "if (!(fl & OC_INIT) || (fl & OC_IDLE)) continue;"),
    "uninitialised_windows_are_candidates": ("if (j == 0 || !(fl & OC_INIT) || (fl & OC_IDLE)) continue;",
                                             "if (j == 0 || (fl & OC_IDLE)) continue;"),
    "n_above_off_by_one": ("best.n_above = N;", "best.n_above = N - 1;"),
    "order_counts_swapped": ("best.concordant += (run_n - run_h) * H;", "best.discordant += (run_n - run_h) * H;"),
    "order_counts_ties": ("best.discordant += run_h * (N - H);", "best.discordant += run_h * (N + run_n - H - run_h);"),
    "order_counts_all_pairs": ("best.concordant += (run_n - run_h) * H;", "best.concordant += (run_n - run_h) * N;"),
}


@pytest.fixture(scope="module")
def tmpdir():
    with tempfile.TemporaryDirectory() as d:
        yield d


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_calib_mutant_is_caught(name, tmpdir):
    old, new = MUTANTS[name]
    text = open(SRC_CALIB).read()
    assert text.count(old) == 1, f"mutant {name}: pattern not unique in the oracle"
    src = os.path.join(tmpdir, f"{name}.c")
    open(src, "w").write(text.replace(old, new))
    lib = os.path.join(tmpdir, f"lib{name}.so")
    subprocess.check_call(["gcc", *O.CFLAGS, "-o", lib, SRC_BASE, src, "-lm"])
    o = O.Oracle(lib)
    failed = []
    for pin in calib_pins.ALL:
        try:
            pin(o)
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passes every pin"
