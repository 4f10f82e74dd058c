"""GPU parity of the control replay with the actuation model
(tre_rebalance_act, tre_sweep_act) against the oracle's actuation replay.

Inputs: the bursty and sweep workloads and hand-shaped traces, with wake /
sleep delays (the paper's 1.31 s / 1.87 s and others, rounded up to whole
windows as the library does), random footprints of 1 to 3 GPUs with the
budget raised to fit, and random per-tick veto masks. Every scenario's move
log, final replicas and replica-window sums must match bit for bit.
"""
import sys

import numpy as np
import pytest

import oracle as O
import tracegen as tg
import edge_traces as E
import parity as PT

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_29160_amd import device, tre
    return tre, device, torch


def _columns(torch, traces):
    counts = [len(t["ts"]) for t in traces]
    off = np.zeros(len(traces) + 1, np.int64)
    off[1:] = np.cumsum(counts)
    n = int(off[-1]) + 16
    cols = {}
    for k, dt in (("ts", np.int64), ("model", np.uint8), ("req", np.uint32), ("type", np.uint8),
                  ("tokens", np.uint16)):
        a = np.zeros(n, dt)
        for i, t in enumerate(traces):
            a[off[i]:off[i + 1]] = t[k]
        cols[k] = torch.from_numpy(a).cuda()
    return cols, off


def _ticks(cfg):
    nW = cfg["duration_ms"] // cfg["window_ms"]
    return [w for w in range(nW) if ((w + 1) * cfg["window_ms"]) % cfg["fast_period_ms"] == 0
            or ((w + 1) * cfg["window_ms"]) % cfg["slow_period_ms"] == 0]


def _ceil_w(ms, cfg):
    nW = cfg["duration_ms"] // cfg["window_ms"]
    return min(-(-ms // cfg["window_ms"]), nW + 1)


def _check(lib, name, cfg, traces, prof_cols, sc_cols, wake_ms, sleep_ms, g=None, veto=None, sweep=True):
    """Both entry points against the oracle for every scenario. g: int32
    [n_traces][M] or None; veto: uint64 [n_traces][n_ticks] or None."""
    tre, device, torch = lib
    M = cfg["n_models"]
    cols, off = _columns(torch, traces)
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
    prof = tre.pack(prof_cols, tre.PROFILE_DTYPE)
    sc = tre.pack(sc_cols, tre.SCENARIO_DTYPE)
    tre.tre_check_params(ev, prof, sc)
    g_t = None if g is None else torch.from_numpy(np.ascontiguousarray(g, np.int32)).cuda()
    v_t = None if veto is None else torch.from_numpy(np.ascontiguousarray(veto, np.uint64).view(np.int64)).cuda()
    act = tre.actuation(wake_ms, sleep_ms, g_t, v_t)
    tre.tre_check_actuation(ev, prof, act)
    n_sc = len(sc_cols["trace"])
    move_cap = max(1, ev.n_ticks * int(np.max(sc_cols["max_moves"])))
    tss = tre.tss_outputs(ev, which=("tss64", "flags"))
    tre.tre_eval_tss(ev, prof, tss)
    outs = []
    out = tre.ctl_outputs(ev, n_sc, move_cap)
    tre.tre_rebalance_act(ev, prof, tss["tss64"], tss["flags"], sc, act, out)
    outs.append(("rebalance_act", out))
    if sweep:
        out2 = tre.ctl_outputs(ev, n_sc, move_cap)
        ws = torch.empty(tre.tre_workspace_size(ev, n_sc), dtype=torch.uint8, device="cuda")
        tre.tre_sweep_act(ev, prof, sc, act, out2, ws)
        outs.append(("sweep_act", out2))
    torch.cuda.synchronize()
    S = tss["tss64"].cpu().numpy()
    fl = tss["flags"].cpu().numpy()
    o = O.get()
    ww, sw = _ceil_w(wake_ms, cfg), _ceil_w(sleep_ms, cfg)
    for s in range(n_sc):
        t = int(sc_cols["trace"][s])
        prof_t = O.pack_profiles(PT.trace_profile(prof_cols, t, M))
        row = np.zeros(1, O.SCENARIO_DTYPE)
        for k in O.SCENARIO_DTYPE.names:
            row[k] = sc_cols[k][s]
        ref = o.control_act(cfg, prof_t, S[t], fl[t], row, ww, sw,
                            footprint=None if g is None else g[t], veto=None if veto is None else veto[t],
                            move_cap=move_cap)
        for how, oo in outs:
            moves = tre.unpack_moves(oo["moves"]).reshape(-1)[s * move_cap:(s + 1) * move_cap]
            PT.compare_ctl(moves, int(oo["n_moves"][s]), oo["r_final"][s].cpu().numpy(),
                           oo["r_windows"][s].cpu().numpy(), ref, f"{name} {how} scenario {s}")
    ev.close()
    return outs


def _random_act(rng, prof_cols, n_traces, M, cfg, veto_p=0.3):
    g = rng.integers(1, 4, (n_traces, M)).astype(np.int32)
    r_init = np.asarray(prof_cols["r_init"]).reshape(n_traces, M)
    budget = int((g * r_init).sum(axis=1).max() + rng.integers(0, 6))
    nt = len(_ticks(cfg))
    full = (1 << M) - 1 if M < 64 else (1 << 64) - 1
    veto = rng.integers(0, 1 << 62, (n_traces, nt), dtype=np.int64).astype(np.uint64)
    veto &= np.uint64(full)
    veto[rng.random((n_traces, nt)) > veto_p] = 0
    return g, budget, veto


def test_instantaneous_actuation_equals_the_plain_calls(lib):
    tre, device, torch = lib
    w = tg.standard(2)
    ev_h = w.generate(0, 1)
    traces = [ev_h.trace(0)]
    sc = w.scenario_columns()
    sc = {k: v[:256] for k, v in sc.items()}
    outs = _check(lib, "sweep256-instant", w.trace_cfg(), traces, w.profile_columns(1), sc, 0, 0,
                  g=np.ones((1, w.n_models), np.int32))
    # and the plain sweep on the same inputs
    cols, off = _columns(torch, traces)
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off,
                             w.trace_cfg())
    prof = tre.pack(w.profile_columns(1), tre.PROFILE_DTYPE)
    sct = tre.pack(sc, tre.SCENARIO_DTYPE)
    cap = outs[0][1]["move_cap"]
    out = tre.ctl_outputs(ev, 256, cap)
    ws = torch.empty(tre.tre_workspace_size(ev, 256), dtype=torch.uint8, device="cuda")
    tre.tre_sweep(ev, prof, sct, out, ws)
    torch.cuda.synchronize()
    for k in ("moves", "n_moves", "r_final", "r_windows"):
        assert torch.equal(out[k], outs[1][1][k]), k
    ev.close()


@pytest.mark.parametrize("wake_ms,sleep_ms", [(1310, 1870), (500, 0), (0, 2500), (7000, 12000)])
def test_bursty_with_delays_footprints_vetoes(lib, wake_ms, sleep_ms):
    w = tg.standard(1)
    traces = [w.generate(0, 1).trace(0)]
    prof = w.profile_columns(1)
    rng = np.random.default_rng(wake_ms + 7 * sleep_ms)
    cfg = dict(w.trace_cfg())
    g, budget, veto = _random_act(rng, prof, 1, w.n_models, cfg)
    cfg["budget"] = budget
    sc = {"trace": np.zeros(12, np.uint32), "max_moves": rng.choice(np.array([1, 2, 4], np.uint32), 12),
          "theta_scale": rng.uniform(0.5, 2.0, 12), "tau_crit_override": np.where(rng.random(12) < 0.5, -1.0,
                                                                                   rng.uniform(0.2, 0.8, 12))}
    say(f"bursty wake {wake_ms} sleep {sleep_ms} budget {budget}")
    _check(lib, f"bursty-{wake_ms}-{sleep_ms}", cfg, traces, prof, sc, wake_ms, sleep_ms, g=g, veto=veto)


def test_sweep_1024_scenarios_with_paper_delays(lib):
    w = tg.standard(2)
    traces = [w.generate(0, 1).trace(0)]
    prof = w.profile_columns(1)
    rng = np.random.default_rng(3)
    cfg = dict(w.trace_cfg())
    g, budget, veto = _random_act(rng, prof, 1, w.n_models, cfg, veto_p=0.1)
    cfg["budget"] = budget
    _check(lib, "sweep1024-act", cfg, traces, prof, w.scenario_columns(), 1310, 1870, g=g, veto=veto)


@pytest.mark.parametrize("M", [1, 5, 33, 64])
def test_model_counts_with_actuation(lib, M):
    win, nW = 250, 1600
    cfg = {"window_ms": win, "duration_ms": win * nW, "fast_period_ms": win * 4, "slow_period_ms": win * 8,
           "n_models": M, "budget": 0}
    traces = [E.trace_random(80 + M + i, M, win * nW, 300 * M) for i in range(3)]
    rng = np.random.default_rng(M)
    n = 3 * M
    prof = {"w_p": rng.uniform(0.05, 0.9, n), "w_q": rng.uniform(1.0, 3.0, n), "alpha": rng.uniform(0.05, 1.0, n),
            "theta": rng.uniform(20.0, 400.0, n), "tau_crit": rng.uniform(0.2, 0.6, n),
            "tau_surplus": rng.uniform(1.1, 2.0, n), "r_min": rng.integers(0, 2, n).astype(np.int32),
            "r_init": np.full(n, 2, np.int32)}
    g, budget, veto = _random_act(rng, prof, 3, M, cfg)
    cfg["budget"] = budget
    sc = {"trace": (np.arange(9) % 3).astype(np.uint32), "max_moves": rng.choice(np.array([1, 2, 4, 8], np.uint32), 9),
          "theta_scale": rng.uniform(0.5, 2.0, 9), "tau_crit_override": -np.ones(9)}
    _check(lib, f"M{M}-act", cfg, traces, prof, sc, int(rng.integers(0, 4000)), int(rng.integers(0, 4000)),
           g=g, veto=veto)


def test_delays_past_the_trace(lib):
    """Transitions that cannot complete before the end never count."""
    w = tg.standard(0)
    traces = [w.generate(0, 1).trace(0)]
    cfg = dict(w.trace_cfg())
    sc = {"trace": np.zeros(3, np.uint32), "max_moves": np.array([1, 2, 4], np.uint32),
          "theta_scale": np.ones(3), "tau_crit_override": -np.ones(3)}
    _check(lib, "tiny-long-delays", cfg, traces, w.profile_columns(1), sc, 10 ** 9, 10 ** 12)


def test_actuation_argument_errors(lib):
    tre, device, torch = lib
    w = tg.standard(0)
    traces = [w.generate(0, 1).trace(0)]
    cols, off = _columns(torch, traces)
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off,
                             w.trace_cfg())
    prof = tre.pack(w.profile_columns(1), tre.PROFILE_DTYPE)
    for g in ([0, 1, 1], [3, 3, 3]):  # a zero footprint; GPUs above the budget of 8
        gt = torch.tensor([g], dtype=torch.int32, device="cuda")
        with pytest.raises(tre.TreError) as e:
            tre.tre_check_actuation(ev, prof, tre.actuation(0, 0, gt))
        assert e.value.code == tre.TRE_EINVAL
    with pytest.raises(tre.TreError) as e:
        tre.tre_check_actuation(ev, prof, tre.actuation(-1, 0))
    assert e.value.code == tre.TRE_EINVAL
    sc = tre.pack(w.scenario_columns(), tre.SCENARIO_DTYPE)
    out = tre.ctl_outputs(ev, 1, 16)
    ws = torch.empty(tre.tre_workspace_size(ev, 1), dtype=torch.uint8, device="cuda")
    with pytest.raises(tre.TreError) as e:
        tre.tre_sweep_act(ev, prof, sc, tre.actuation(0, -5), out, ws)
    assert e.value.code == tre.TRE_EINVAL
    ev.close()
