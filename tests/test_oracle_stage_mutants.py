"""Pin strength of the stage-aware service-share oracle: plausible mistakes
planted in copies of ``oracle/tre_oracle_stage.c`` (compiled on the CPU
together with the unmodified base oracle) must each fail at least one pin
of stage_pins.py."""
import os
import subprocess
import tempfile

import pytest

import oracle as O
import stage_pins

HERE = os.path.dirname(O.__file__)
SRC_STAGE = os.path.join(HERE, "tre_oracle_stage.c")
SRC_BASE = os.path.join(HERE, "tre_oracle.c")

MUTANTS = {
    "prefill_weight_dropped": ("double num = w_p * (double)P;", "double num = (double)P;"),
    "waiting_weight_dropped": ("double den = w_q * (double)W_int;", "double den = (double)W_int;"),
    "prefill_floor_dropped": ("  if (den < (double)window_ms) den = (double)window_ms;\n  return num / den;\n}\n\n/* raw decode",
                              "  return num / den;\n}\n\n/* raw decode"),
    "decode_floor_dropped": ("  double den = (double)A_int;\n  if (den < (double)window_ms) den = (double)window_ms;",
                             "  double den = (double)A_int;"),
    "prefill_over_active": ("oracle_stage_raw_prefill(prof[m].w_p, prof[m].w_q, P[c], W_int[c], window_ms)",
                            "oracle_stage_raw_prefill(prof[m].w_p, prof[m].w_q, P[c], A_int[c], window_ms)"),
    "decode_counts_prompt": ("oracle_stage_raw_decode(D[c], A_int[c], window_ms)", "oracle_stage_raw_decode(P[c], A_int[c], window_ms)"),
    "prefill_idle_ignores_waiting": ("const int p_idle = P[c] == 0 && W_int[c] == 0;", "const int p_idle = P[c] == 0;"),
    "decode_idle_ignores_active": ("const int d_idle = D[c] == 0 && A_int[c] == 0;", "const int d_idle = D[c] == 0;"),
    "decode_init_from_zero": ("          sd = raw;\n          id = 1;", "          sd = prof[m].alpha * raw;\n          id = 1;"),
    "prefill_alpha_swapped": ("          const double t1 = prof[m].alpha * raw;\n          const double t2 = (1.0 - prof[m].alpha) * sp;",
                              "          const double t1 = (1.0 - prof[m].alpha) * raw;\n          const double t2 = prof[m].alpha * sp;"),
    "init_flags_swapped": ("(ip ? OS_P_INIT : 0) | (d_idle ? OS_D_IDLE : 0) |\n                           (id ? OS_D_INIT : 0)",
                           "(id ? OS_P_INIT : 0) | (d_idle ? OS_D_IDLE : 0) |\n                           (ip ? OS_D_INIT : 0)"),
    "decode_rate_per_ms": ("double num = (double)D * 1000.0;", "double num = (double)D;"),
    "stages_swapped_in_output": ("      S[2 * c] = sp;\n      S[2 * c + 1] = sd;", "      S[2 * c] = sd;\n      S[2 * c + 1] = sp;"),
}


@pytest.fixture(scope="module")
def tmpdir():
    with tempfile.TemporaryDirectory() as d:
        yield d


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_stage_mutant_is_caught(name, tmpdir):
    old, new = MUTANTS[name]
    text = open(SRC_STAGE).read()
    assert text.count(old) == 1, f"mutant {name}: pattern not unique in the oracle"
    src = os.path.join(tmpdir, f"{name}.c")
    open(src, "w").write(text.replace(old, new))
    lib = os.path.join(tmpdir, f"lib{name}.so")
    subprocess.check_call(["gcc", *O.CFLAGS, "-o", lib, SRC_BASE, src, "-lm"])
    o = O.Oracle(lib)
    failed = []
    for pin in stage_pins.ALL:
        try:
            pin(o)
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passes every pin"
