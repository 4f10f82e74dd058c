"""GPU parity in every launch shape of the streaming kernel.

``tre_eval_tss`` / ``tre_sweep`` stream one trace per workgroup and size the
workgroup by the number of traces in the handle: 16 waves up to 384 traces,
8 waves up to 768, 4 waves above (the shape the full stress workload runs
in). The tiles are 4096, 2048 and 1024 rows, so the same trace is tallied
with different tile boundaries, deferrals past the LDS ring and evaluation
chunks in each shape. These tests load stress-shaped traces (32 models,
250 ms windows, synchronized flash crowds) in handles of 8, 400 and 800
traces and compare

  * every per-cell output of ``tre_eval_tss`` (prefill, decode, A_int,
    W_int, fp64 TSS bit for bit, fp32 TSS, flags) of every trace, and every
    scenario's control outputs from ``tre_rebalance`` and from ``tre_sweep``
    (with and without the fp32 TSS, which take different kernel
    instantiations), with the CPU oracle;
  * the first 8 traces across the three handles: identical bytes.
"""
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle as O
import tracegen as tg
import parity as PT

pytestmark = pytest.mark.gpu

N_MAX = 800
DURATION_MS = 60_000


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _workload(n):
    # flash crowds every 20 s (four models at 10x for 5 s), so some windows
    # are dense enough for a 4096-row tile to reach past the ring
    return tg.standard(4).scaled(n_traces=n, n_scenarios=n, duration_ms=DURATION_MS, proc_params={
        "flash_mult": 10.0, "flash_len_s": 5.0, "flash_first_s": 10.0, "flash_every_s": 20.0, "flash_models": 4})


def _scenarios(n):
    """Scenario s runs on trace s: the first n rows of one table, so the
    first 8 scenarios are the same in every handle."""
    rng = np.random.default_rng(2024)
    cols = {"trace": np.arange(N_MAX, dtype=np.uint32),
            "max_moves": rng.choice(np.array([1, 2, 4], np.uint32), N_MAX).astype(np.uint32),
            "theta_scale": rng.uniform(0.5, 2.0, N_MAX),
            "tau_crit_override": np.where(rng.random(N_MAX) < 0.25, -1.0, rng.uniform(0.2, 0.8, N_MAX))}
    return {k: v[:n] for k, v in cols.items()}


@pytest.fixture(scope="module")
def reference():
    """Oracle TSS of traces [0, 800) and the control replay of their
    scenarios (one oracle call per trace on a thread pool)."""
    w = _workload(N_MAX)
    ev = w.generate(0, N_MAX)
    prof = O.pack_profiles(w.profile_columns())
    M = w.n_models
    sc = O.pack_scenarios(_scenarios(N_MAX))
    move_cap = (DURATION_MS // w.window_ms) * 4
    o = O.get()

    def one(t):
        r = o.tss_trace(ev.trace(t), w.window_ms, w.duration_ms, prof[t * M:(t + 1) * M])
        r["ctl"] = o.control(w.trace_cfg(), prof[t * M:(t + 1) * M], r["S"], r["flags"], sc[t:t + 1], move_cap)
        return r

    with ThreadPoolExecutor(max_workers=tg.default_threads()) as pool:
        refs = list(pool.map(one, range(N_MAX)))
    say(f"oracle: {ev.n_events} events in {N_MAX} traces")
    return {"refs": refs, "move_cap": move_cap, "events": ev.n_events}


def _run(n):
    """Load the first n traces, evaluate every per-cell output, replay the
    scenarios from the cells and in the sweep (twice: with and without
    the fp32 TSS). Returns host copies."""
    import torch

    from paper_2609_29160_amd import device, tre

    w = _workload(n)
    dt = device.upload(w)
    ev = device.load(dt, validate=True)
    prof = device.profiles(w)
    sc_cols = _scenarios(n)
    sc = device.scenarios(sc_cols)
    tre.tre_check_params(ev, prof, sc)
    move_cap = (DURATION_MS // w.window_ms) * 4
    say(f"{n} traces: {dt.n_events} events")
    out = tre.tss_outputs(ev)
    tre.tre_eval_tss(ev, prof, out)
    cells = {k: v.cpu().numpy() for k, v in out.items()}
    cells["prefill"] = cells["prefill"].view(np.uint32)
    cells["decode"] = cells["decode"].view(np.uint32)
    ctl = {}
    o1 = tre.ctl_outputs(ev, n, move_cap)
    tre.tre_rebalance(ev, prof, out["tss64"], out["flags"], sc, o1)
    ctl["rebalance"] = o1
    ws = torch.empty(tre.tre_workspace_size(ev, n), dtype=torch.uint8, device="cuda")
    o2 = tre.ctl_outputs(ev, n, move_cap)
    tre.tre_sweep(ev, prof, sc, o2, ws)
    ctl["sweep"] = o2
    o3 = tre.ctl_outputs(ev, n, move_cap)
    t32 = torch.empty((ev.n_traces, ev.n_windows, ev.n_models), dtype=torch.float32, device="cuda")
    tre.tre_sweep(ev, prof, sc, o3, ws, tss32=t32)
    ctl["sweep_tss32"] = o3
    torch.cuda.synchronize()
    host_ctl = {how: {"moves": tre.unpack_moves(o["moves"]).reshape(n, move_cap).copy(),
                      "n_moves": o["n_moves"].cpu().numpy().copy(), "r_final": o["r_final"].cpu().numpy().copy(),
                      "r_windows": o["r_windows"].cpu().numpy().copy()} for how, o in ctl.items()}
    res = {"cells": cells, "ctl": host_ctl, "sweep_tss32": t32.cpu().numpy(), "n_events": dt.n_events}
    ev.close()
    del dt, out, ws, t32
    torch.cuda.empty_cache()
    return res


_cache = {}


def _result(n):
    if n not in _cache:
        _cache[n] = _run(n)
    return _cache[n]


@pytest.mark.parametrize("n", [400, 800])
def test_every_cell_and_scenario(reference, n):
    """8-wave (400 traces) and 4-wave (800 traces) workgroups: every cell of
    every trace and every scenario equal to the oracle."""
    r = _result(n)
    refs = reference["refs"]
    move_cap = reference["move_cap"]
    for t in range(n):
        PT.compare_tss({k: v[t] for k, v in r["cells"].items()}, refs[t], f"{n} traces: trace {t}")
        PT.compare_tss32(r["sweep_tss32"][t], refs[t]["S"], f"{n} traces: sweep tss32 trace {t}")
    moved = 0
    for how, c in r["ctl"].items():
        for s in range(n):
            PT.compare_ctl(c["moves"][s], int(c["n_moves"][s]), c["r_final"][s], c["r_windows"][s],
                           refs[s]["ctl"], f"{n} traces: {how} scenario {s}")
            moved += int(c["n_moves"][s] > 0)
    say(f"{n} traces: {r['n_events']} events, every cell and {n} scenarios x 3 replays match the oracle "
        f"({moved} replays with moves)")
    assert moved > 0


def test_vary_grid():
    """The first 8 traces alone (16-wave workgroups), inside the 400-trace
    handle (8 waves) and inside the 800-trace handle (4 waves): identical
    bytes in every per-cell output and every control output."""
    small = _result(8)
    for n in (400, 800):
        big = _result(n)
        for k, v in small["cells"].items():
            assert np.array_equal(v.view(np.uint8), big["cells"][k][:8].view(np.uint8)), f"{k}: 8 vs {n} traces"
        assert np.array_equal(small["sweep_tss32"].view(np.uint32), big["sweep_tss32"][:8].view(np.uint32))
        for how, c in small["ctl"].items():
            for k, v in c.items():
                got = big["ctl"][how][k][:8]
                assert np.array_equal(np.asarray(v).view(np.uint8), np.asarray(got).view(np.uint8)), \
                    f"{how} {k}: 8 vs {n} traces"
    say("vary grid: 16-, 8- and 4-wave workgroups give identical bytes")
