"""GPU parity at full size, in the launch configuration the benchmark times.

The stress workload (4096 traces x 32 models, 3600 s in 250 ms windows,
9.36e9 events, 150 GB of columns) and the diverse workload (256 traces x 16
models, 7200 s in 1 s windows, 1.57e9 events) are uploaded whole and swept
three times: the three results must be identical (the kernels share LDS
between waves; a missing barrier shows up as launch-to-launch differences
only at this scale), and sampled scenarios and per-cell fp32 TSS of sampled
traces must match the CPU oracle exactly. The oracle regenerates each
sampled trace on the host from the same seeds. The calibration sweep, the
stage-aware shares and the closed-loop replay of the whole stress workload
(with and without the actuation model) are run twice each and checked the
same way (sampled traces or scenarios against the oracle).
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
    tre.tre_calib_order(ev, slo, tss["tss64"], tss["flags"], out)
    fit = tre.unpack_fit(out["fit"]).reshape(T, M)
    fit0 = runs[0][1].view(tre.FIT_DTYPE).reshape(T, M)
    for k in ("theta", "n_cand", "n_healthy", "n_above", "healthy_above"):
        assert np.array_equal(np.ascontiguousarray(fit0[k]).view(np.uint8), np.ascontiguousarray(fit[k]).view(np.uint8)), k
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
        for k in ("n_cand", "n_healthy", "n_above", "healthy_above", "concordant", "discordant"):
            assert np.array_equal(fit[t][k], r["fit"][k]), (t, k)
    say(f"{w.name}: calibration of {len(sample)} sampled traces matches the oracle")
    ev.close()
    del tss, out, dt
    torch.cuda.empty_cache()


def test_stress_full_size_stage_shares():
    """Tallies and stage-aware shares over the whole stress workload, twice:
    identical results, and the shares and flags of sampled traces equal to
    the oracle's bit for bit; then the one-pass path (tre_eval_stage), equal
    to them in every cell."""
    import torch

    from paper_2609_29160_amd import device, tre

    w = tg.standard(4)
    say(f"{w.name}: uploading")
    dt = device.upload(w)
    ev = device.load(dt, validate=True)
    prof = device.profiles(w)
    T, M = ev.n_traces, ev.n_models
    tal = tre.tss_outputs(ev, which=("prefill", "decode", "a_int", "w_int"))
    out = tre.stage_outputs(ev, which=("stage64", "flags"))
    runs = []
    for _ in range(2):
        tre.tre_eval_tss(ev, prof, tal)
        tre.tre_stage_tss(ev, prof, tal, out)
        torch.cuda.synchronize()
        runs.append({k: v.cpu().numpy().copy() for k, v in out.items()})
    for k in runs[0]:
        assert np.array_equal(runs[0][k].view(np.uint8), runs[1][k].view(np.uint8)), f"{k} differs between launches"
    rng = np.random.default_rng(19)
    sample = sorted({0, T - 1, *rng.integers(0, T, 4).tolist()})
    o = PT.O.get()
    prof_all = PT.O.pack_profiles(w.profile_columns())
    for t in sample:
        host = w.generate(t, t + 1).trace(0)
        p = prof_all[t * M:(t + 1) * M]
        r = o.stage_tss(o.tss_trace(host, w.window_ms, w.duration_ms, p), w.window_ms, p)
        assert np.array_equal(runs[0]["stage64"][t].view(np.uint64), r["S"].view(np.uint64)), t
        assert np.array_equal(runs[0]["flags"][t], r["flags"]), t
    say(f"{w.name}: stage shares of {len(sample)} sampled traces match the oracle")
    # the one-pass path: equal to the two-pass shares everywhere
    del tal
    torch.cuda.empty_cache()
    fused = tre.stage_outputs(ev, which=("stage64", "flags"))
    tre.tre_eval_stage(ev, prof, fused)
    torch.cuda.synchronize()
    assert torch.equal(fused["stage64"].view(torch.int64), out["stage64"].view(torch.int64)), "one-pass shares differ"
    assert torch.equal(fused["flags"], out["flags"]), "one-pass flags differ"
    say(f"{w.name}: one-pass stage shares equal the two-pass ones in every cell")
    ev.close()
    del out, fused, dt
    torch.cuda.empty_cache()


_STRESS_TABLES = {}


@pytest.mark.parametrize("actuation", [False, True], ids=["plain", "actuation"])
def test_stress_full_size_closed_loop(actuation):
    """The closed loop over every scenario of the stress workload (777 M
    requests), twice: identical results; sampled scenarios equal to the
    oracle's closed-loop replay (moves, replicas, replica-window sums,
    latency statistics) with no event beyond the ring. With the actuation
    model: the paper's wake and sleep times (1.31 s, 1.87 s), footprints of
    1 or 2 GPUs per replica with the GPU budget at the largest initial
    footprint sum plus 8, vetoes on 10% of the ticks."""
    from concurrent.futures import ThreadPoolExecutor

    import torch

    from paper_2609_29160_amd import tre

    w = tg.standard(4)
    T, M = w.n_traces, w.n_models
    if w.name not in _STRESS_TABLES:
        with ThreadPoolExecutor(max_workers=16) as pool:
            _STRESS_TABLES[w.name] = list(pool.map(w.requests, range(T)))
    tables = _STRESS_TABLES[w.name]
    say(f"{w.name}: {sum(len(t['arrival_ms']) for t in tables)} requests")
    svc = np.zeros(T * M, tre.SERVICE_DTYPE)
    for k, v in w.service_columns().items():
        svc[k] = v
    slo = np.zeros(T * M, tre.SLO_DTYPE)
    for k, v in w.slo_columns().items():
        slo[k] = v
    rq, keep = tre.loop_requests(tables, M, svc, slo)
    cfg = w.trace_cfg()
    prof = tre.pack(w.profile_columns(), tre.PROFILE_DTYPE)
    sc_cols = w.scenario_columns()
    n_sc = len(sc_cols["trace"])
    sc = tre.pack(sc_cols, tre.SCENARIO_DTYPE)
    nW = w.n_windows
    n_ticks = sum(1 for x in range(nW) if ((x + 1) * w.window_ms) % cfg["fast_period_ms"] == 0
                  or ((x + 1) * w.window_ms) % cfg["slow_period_ms"] == 0)
    move_cap = max(1, n_ticks * int(np.max(sc_cols["max_moves"])))

    class _Shape:
        n_models = M

    kw_t = lambda t: {}
    if actuation:
        rng = np.random.default_rng(31)
        fp = rng.integers(1, 3, (T, M)).astype(np.int32)
        r_init = np.asarray(w.profile_columns()["r_init"]).reshape(T, M)
        cfg = dict(cfg, budget=int((fp * r_init).sum(axis=1).max()) + 8)
        veto = np.frombuffer(rng.bytes(8 * T * n_ticks), np.uint64).reshape(T, n_ticks).copy()
        veto &= np.uint64((1 << M) - 1)
        veto[rng.random(veto.shape) >= 0.1] = 0
        g_dev = torch.from_numpy(fp).cuda()
        v_dev = torch.from_numpy(veto.view(np.int64)).cuda()
        act = tre.actuation(1310, 1870, g_dev, v_dev)
        to_w = lambda ms: min(-(-ms // w.window_ms), nW + 1)
        kw_t = lambda t: {"wake_w": to_w(1310), "sleep_w": to_w(1870), "footprint": fp[t], "veto": veto[t]}
    ws = torch.empty(tre.tre_loop_workspace_size(cfg, rq, n_sc), dtype=torch.uint8, device="cuda")
    runs = []
    for _ in range(2):
        out = tre.ctl_outputs(_Shape(), n_sc, move_cap)
        stats = torch.zeros(n_sc * M * tre.LOOP_STATS_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
        if actuation:
            tre.tre_loop_act(cfg, T, rq, prof, sc, act, out, stats, ws)
        else:
            tre.tre_loop(cfg, T, rq, prof, sc, out, stats, ws)
        torch.cuda.synchronize()
        assert int(ws[:8].cpu().numpy().view(np.uint64)[0]) == 0, "events beyond the ring"
        runs.append((_outputs(out), stats.cpu().numpy().copy()))
    for k in runs[0][0]:
        assert np.array_equal(runs[0][0][k], runs[1][0][k]), f"{k} differs between launches"
    assert np.array_equal(runs[0][1], runs[1][1]), "statistics differ between launches"
    o = PT.O.get()
    prof_all = PT.O.pack_profiles(w.profile_columns())
    slo_all = PT.O.pack_slo(w.slo_columns())
    svc_all = PT.O.pack_svc(w.service_columns())
    sc_all = PT.O.pack_scenarios(sc_cols)
    rng = np.random.default_rng(23)
    sample = sorted({0, n_sc - 1, *rng.integers(0, n_sc, 2).tolist()})

    def one(s):
        t = int(sc_all[s]["trace"])
        return o.loop(cfg, prof_all[t * M:(t + 1) * M], sc_all[s:s + 1], slo_all[t * M:(t + 1) * M],
                      svc_all[t * M:(t + 1) * M], tables[t], move_cap=move_cap, **kw_t(t))

    say(f"{w.name}: oracle closed loop of scenarios {sample}")
    with ThreadPoolExecutor(max_workers=len(sample)) as pool:
        refs = list(pool.map(one, sample))
    g, st = runs[0]
    moves = tre.unpack_moves(torch.from_numpy(g["moves"])).reshape(n_sc, move_cap)
    st = st.view(tre.LOOP_STATS_DTYPE).reshape(n_sc, M)
    for s, ref in zip(sample, refs):
        n = int(g["n_moves"][s])
        assert n == ref["n_moves"], (s, n, ref["n_moves"])
        k = min(n, move_cap)
        for f in ("window", "path", "receiver", "donor"):
            assert np.array_equal(moves[s][:k][f], ref["moves"][:k][f]), (s, f)
        assert np.array_equal(g["r_final"][s], ref["r_final"]), s
        assert np.array_equal(g["r_windows"][s], ref["r_windows"]), s
        for f in tre.LOOP_STATS_DTYPE.names:
            assert np.array_equal(st[s][f], ref["stats"][f]), (s, f)
    assert sum(int(g["n_moves"][s]) for s in sample) > 0, "no moves in the sampled scenarios"
    say(f"{w.name}: closed loop of {len(sample)} sampled scenarios matches the oracle")
    if actuation:  # the last variant: free the host tables
        _STRESS_TABLES.clear()
