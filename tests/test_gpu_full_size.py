"""GPU parity at full size, in the launch configuration the benchmark times.

The stress workload (4096 traces x 32 models, 3600 s in 250 ms windows,
9.36e9 events, 150 GB of columns) and the diverse workload (256 traces x 16
models, 7200 s in 1 s windows, 1.57e9 events) are uploaded whole and swept
three times: the three results must be identical (the kernels share LDS
between waves; a missing barrier shows up as launch-to-launch differences
only at this scale), and sampled scenarios and per-cell fp32 TSS of sampled
traces must match the CPU oracle exactly. The oracle regenerates each
sampled trace on the host from the same seeds.
"""
import sys

import numpy as np
import pytest

import tracegen as tg
import parity as PT

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _outputs(out):
    return {k: out[k].cpu().numpy().copy() for k in ("moves", "n_moves", "r_final", "r_windows")}


def _run_full(workload_index, sample_traces, tss_traces, act_seed=None):
    """act_seed: run with the actuation model (the paper's 1.31 s wake and
    1.87 s sleep, footprints of 1 or 2 GPUs drawn from the seed, the budget
    raised to fit with 8 GPUs to spare, vetoes on 10% of the ticks)."""
    import torch

    from paper_2609_29160_amd import device, tre

    w = tg.standard(workload_index)
    say(f"{w.name}: uploading")
    dt = device.upload(w)
    cfg = dict(w.trace_cfg())
    M = w.n_models
    act = g = veto = None
    if act_seed is not None:
        rng = np.random.default_rng(act_seed)
        g = rng.integers(1, 3, (w.n_traces, M)).astype(np.int32)
        r_init = np.asarray(w.profile_columns()["r_init"]).reshape(w.n_traces, M)
        cfg["budget"] = int((g * r_init).sum(axis=1).max()) + 8
    c = dt.cols
    ev = tre.tre_load_events(c["ts"], c["model"], c["req"], c["type"], c["tokens"], dt.off, cfg, validate=True)
    prof = device.profiles(w)
    if act_seed is not None:
        veto = rng.integers(0, 1 << 62, (w.n_traces, ev.n_ticks), dtype=np.int64).astype(np.uint64)
        veto &= np.uint64((1 << M) - 1)
        veto[rng.random(veto.shape) > 0.1] = 0
        g_t = torch.from_numpy(g).cuda()
        v_t = torch.from_numpy(veto.view(np.int64)).cuda()
        act = tre.actuation(1310, 1870, g_t, v_t)
        tre.tre_check_actuation(ev, prof, act)
    sweep = (lambda **kw: tre.tre_sweep(ev, prof, sc, out, ws, **kw)) if act is None else \
        (lambda **kw: tre.tre_sweep_act(ev, prof, sc, act, out, ws, **kw))
    sc_cols = w.scenario_columns()
    n_sc = len(sc_cols["trace"])
    sc = device.scenarios(sc_cols)
    tre.tre_check_params(ev, prof, sc)
    move_cap = max(1, ev.n_ticks * int(np.max(sc_cols["max_moves"])))
    out = tre.ctl_outputs(ev, n_sc, move_cap)
    ws = torch.empty(tre.tre_workspace_size(ev, n_sc), dtype=torch.uint8, device="cuda")
    say(f"{w.name}: {dt.n_events} events, {n_sc} scenarios; three sweeps")
    runs = []
    for _ in range(3):
        sweep()
        torch.cuda.synchronize()
        runs.append(_outputs(out))
    for r in runs[1:]:
        for k in runs[0]:
            assert np.array_equal(runs[0][k], r[k]), f"{w.name}: sweep output {k} differs between launches"
    # the same launch with the per-cell fp32 TSS written
    t32 = torch.empty((ev.n_traces, ev.n_windows, ev.n_models), dtype=torch.float32, device="cuda")
    sweep(tss32=t32)
    torch.cuda.synchronize()
    with_tss = _outputs(out)
    for k in runs[0]:
        assert np.array_equal(runs[0][k], with_tss[k]), f"{w.name}: emitting TSS changed {k}"

    prof_all = PT.O.pack_profiles(w.profile_columns())
    by_trace = {}
    for s, t in enumerate(sc_cols["trace"]):
        by_trace.setdefault(int(t), []).append(s)
    moves = tre.unpack_moves(out["moves"]).reshape(n_sc, move_cap)
    checked = 0
    for t in sorted(set(sample_traces) | set(tss_traces)):
        host = w.generate(t, t + 1).trace(0)
        ref = PT.O.get().tss_trace(host, w.window_ms, w.duration_ms, prof_all[t * M:(t + 1) * M])
        if t in tss_traces:
            PT.compare_tss32(t32[t].cpu().numpy(), ref["S"], f"{w.name} trace {t} tss32")
        if t in sample_traces:
            for s in by_trace.get(t, []):
                row = {k: v[s] for k, v in sc_cols.items()}
                if act is None:
                    exp = PT.oracle_control(w, PT.trace_profile(w.profile_columns(t + 1), t, M), ref["S"],
                                            ref["flags"], row, move_cap)
                else:
                    r1 = np.zeros(1, PT.O.SCENARIO_DTYPE)
                    for k in PT.O.SCENARIO_DTYPE.names:
                        r1[k] = row[k]
                    win = cfg["window_ms"]
                    exp = PT.O.get().control_act(cfg, prof_all[t * M:(t + 1) * M], ref["S"], ref["flags"], r1,
                                                 -(-1310 // win), -(-1870 // win), footprint=g[t], veto=veto[t],
                                                 move_cap=move_cap)
                PT.compare_ctl(moves[s], int(runs[0]["n_moves"][s]), runs[0]["r_final"][s],
                               runs[0]["r_windows"][s], exp, f"{w.name} scenario {s}")
                checked += 1
    say(f"{w.name}: {checked} scenarios and {len(tss_traces)} traces of TSS match the oracle")
    assert checked > 0
    ev.close()


def test_stress_full_size():
    rng = np.random.default_rng(11)
    sample = sorted({0, 1, 2047, 4095, *rng.integers(0, 4096, 4).tolist()})
    _run_full(4, sample, [0, 4095])


def test_stress_full_size_with_actuation():
    rng = np.random.default_rng(13)
    sample = sorted({0, 4095, *rng.integers(0, 4096, 3).tolist()})
    _run_full(4, sample, [], act_seed=14)


def test_diverse_full_size():
    rng = np.random.default_rng(12)
    sample = sorted({0, 255, *rng.integers(0, 256, 3).tolist()})
    _run_full(3, sample, [0, 255])


def test_stress_full_size_calibration():
    """The calibration sweep over the whole stress workload (every trace's
    request table and fit in one launch each), twice: identical results, and
    the counts and fits of sampled traces equal to the oracle's."""
    import torch

    from paper_2609_29160_amd import device, tre

    w = tg.standard(4)
    say(f"{w.name}: uploading")
    dt = device.upload(w)
    ev = device.load(dt, validate=True)
    prof = device.profiles(w)
    slo = device.slos(w)
    T, M, nW = ev.n_traces, ev.n_models, ev.n_windows
    tss = {"tss64": torch.empty((T, nW, M), dtype=torch.float64, device="cuda"),
           "flags": torch.empty((T, nW, M), dtype=torch.uint8, device="cuda")}
    out = tre.calib_outputs(ev, dt.req_cap)
    say(f"{w.name}: {dt.n_events} events, req_cap {dt.req_cap}; two calibration sweeps")
    runs = []
    for _ in range(2):
        tre.tre_eval_tss(ev, prof, tss)
        tre.tre_calibrate(ev, slo, tss["tss64"], tss["flags"], out)
        torch.cuda.synchronize()
        runs.append((out["counts"].cpu().numpy().copy(), out["fit"].cpu().numpy().copy(),
                     int(out["n_bad"].cpu().numpy()[0])))
    assert np.array_equal(runs[0][0], runs[1][0]), "counts differ between launches"
    assert np.array_equal(runs[0][1], runs[1][1]), "fits differ between launches"
    assert runs[0][2] == 0
    counts = runs[0][0].view(np.uint32)
    fit = runs[0][1].view(tre.FIT_DTYPE).reshape(T, M)
    rng = np.random.default_rng(17)
    sample = sorted({0, T - 1, *rng.integers(0, T, 4).tolist()})
    o = PT.O.get()
    prof_all = PT.O.pack_profiles(w.profile_columns())
    slo_all = PT.O.pack_slo(w.slo_columns())
    for t in sample:
        host = w.generate(t, t + 1).trace(0)
        r = o.calibrate(host, w.window_ms, w.duration_ms, prof_all[t * M:(t + 1) * M], slo_all[t * M:(t + 1) * M],
                        dt.req_cap)
        assert np.array_equal(counts[t] >> 16, r["judged"]) and np.array_equal(counts[t] & 0xFFFF, r["ok"]), t
        assert np.array_equal(fit[t]["theta"].view(np.uint64), r["fit"]["theta"].view(np.uint64)), t
        for k in ("n_cand", "n_healthy", "n_above", "healthy_above"):
            assert np.array_equal(fit[t][k], r["fit"][k]), (t, k)
    say(f"{w.name}: calibration of {len(sample)} sampled traces matches the oracle")
    ev.close()
    del tss, out, dt
    torch.cuda.empty_cache()
