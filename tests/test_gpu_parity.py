"""GPU parity: the HIP library against the CPU oracle on the same inputs.

Every test here runs the kernels through the C ABI (ctypes binding) and
compares element by element (small and medium inputs spanning many tiles,
ragged tails and edge cases) or on sampled traces (full-size workloads).
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


def _columns_from_host(torch, traces, pad_front=0, pad_back=0):
    """Concatenate host traces into device columns; returns cols, offsets.
    Columns keep 16 readable rows past the last one (the ABI's requirement)
    plus `pad_back` more."""
    counts = [len(t["ts"]) for t in traces]
    off = np.zeros(len(traces) + 1, np.int64)
    off[0] = pad_front
    off[1:] = pad_front + np.cumsum(counts)
    n = int(off[-1]) + 16 + pad_back
    cols = {}
    for k, dt in (("ts", np.int64), ("model", np.uint8), ("req", np.uint32), ("type", np.uint8),
                  ("tokens", np.uint16)):
        a = np.zeros(max(n, 1), dt)
        for i, t in enumerate(traces):
            a[off[i]:off[i + 1]] = t[k]
        cols[k] = torch.from_numpy(a).cuda()
    return cols, off


def _eval_all(tre, ev, prof):
    out = tre.tss_outputs(ev)
    tre.tre_eval_tss(ev, prof, out)
    host = {k: v.cpu().numpy() for k, v in out.items()}
    host["prefill"] = host["prefill"].view(np.uint32)
    host["decode"] = host["decode"].view(np.uint32)
    return host


def _check_set(lib, name, cfg, traces, prof_cols, sc_cols, pad_front=0, pad_back=0, sweep=True):
    """Full elementwise parity of eval, rebalance and sweep on a trace set."""
    tre, device, torch = lib
    M = cfg["n_models"]
    cols, off = _columns_from_host(torch, traces, pad_front, pad_back)
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
    prof = tre.pack(prof_cols, tre.PROFILE_DTYPE)
    sc = tre.pack(sc_cols, tre.SCENARIO_DTYPE)
    tre.tre_check_params(ev, prof, sc)
    g = _eval_all(tre, ev, prof)

    class W:  # the oracle helpers want window / duration
        window_ms = cfg["window_ms"]
        duration_ms = cfg["duration_ms"]

        @staticmethod
        def trace_cfg():
            return cfg

    refs = []
    for t, tr in enumerate(traces):
        ref = PT.oracle_tss(tr, W, PT.trace_profile(prof_cols, t, M))
        refs.append(ref)
        PT.compare_tss({k: v[t] for k, v in g.items()}, ref, f"{name} trace {t}")
    n_sc = len(sc_cols["trace"])
    move_cap = max(1, ev.n_ticks * int(np.max(sc_cols["max_moves"])))
    outs = []
    out = tre.ctl_outputs(ev, n_sc, move_cap)
    tre.tre_rebalance(ev, prof, torch.from_numpy(g["tss64"]).cuda(), torch.from_numpy(g["flags"]).cuda(), sc, out)
    outs.append(("rebalance", out))
    if sweep:
        out2 = tre.ctl_outputs(ev, n_sc, move_cap)
        ws = torch.empty(tre.tre_workspace_size(ev, n_sc), dtype=torch.uint8, device="cuda")
        t32 = torch.empty((ev.n_traces, ev.n_windows, M), dtype=torch.float32, device="cuda")
        tre.tre_sweep(ev, prof, sc, out2, ws, tss32=t32)
        outs.append(("sweep", out2))
        t32h = t32.cpu().numpy()
        for t in range(len(traces)):
            PT.compare_tss32(t32h[t], refs[t]["S"], f"{name} sweep tss32 trace {t}")
    torch.cuda.synchronize()
    for s in range(n_sc):
        t = int(sc_cols["trace"][s])
        row = {k: v[s] for k, v in sc_cols.items()}
        ref = PT.oracle_control(W, PT.trace_profile(prof_cols, t, M), refs[t]["S"], refs[t]["flags"], row,
                                move_cap)
        for how, o in outs:
            moves = tre.unpack_moves(o["moves"]).reshape(-1)[s * move_cap:(s + 1) * move_cap]
            PT.compare_ctl(moves, int(o["n_moves"][s]), o["r_final"][s].cpu().numpy(),
                           o["r_windows"][s].cpu().numpy(), ref, f"{name} {how} scenario {s}")
    ev.close()
    return refs


def _workload_set(w, t0, t1, sc_cols=None):
    evs = w.generate(t0, t1, threads=8)
    traces = [evs.trace(i) for i in range(t1 - t0)]
    prof_cols = w.profile_columns(t1 - t0)
    if sc_cols is None:
        sc_cols = w.scaled(n_traces=t1 - t0).scenario_columns() if w.scenario_seed is None else None
    return traces, prof_cols, sc_cols


def _random_scenarios(n_traces, n, seed):
    rng = np.random.default_rng(seed)
    return {"trace": (np.arange(n) % n_traces).astype(np.uint32),
            "max_moves": rng.choice(np.array([1, 2, 4, 8], np.uint32), n).astype(np.uint32),
            "theta_scale": rng.uniform(0.5, 2.0, n), "tau_crit_override": np.where(rng.random(n) < 0.5, -1.0, rng.uniform(0.2, 0.8, n))}


# ------------------------------------------------------ standard workloads
def test_tiny_3_models(lib):
    w = tg.standard(0)
    traces, prof, _ = _workload_set(w, 0, 1)
    say("tiny: events", len(traces[0]["ts"]))
    sc = _random_scenarios(1, 16, 1)
    sc["trace"][:] = 0
    sc0 = w.scenario_columns()
    sc = {k: np.concatenate([sc0[k].astype(sc[k].dtype), sc[k]]) for k in sc}
    _check_set(lib, "tiny", w.trace_cfg(), traces, prof, sc)


def test_bursty_8_models(lib):
    w = tg.standard(1)
    traces, prof, sc = _workload_set(w, 0, 1)
    say("bursty: events", len(traces[0]["ts"]))
    _check_set(lib, "bursty", w.trace_cfg(), traces, prof, sc)


def test_sweep_1024_scenarios_on_one_trace(lib):
    w = tg.standard(2)
    traces, prof, _ = _workload_set(w, 0, 1)
    sc = w.scenario_columns()
    say("sweep-1024: scenarios", len(sc["trace"]))
    _check_set(lib, "sweep1024", w.trace_cfg(), traces, prof, sc)


def test_diverse_16_models_short(lib):
    w = tg.standard(3).scaled(duration_ms=900_000, n_traces=4)
    traces, prof, _ = _workload_set(w, 0, 4)
    sc = _random_scenarios(4, 12, 3)
    say("diverse-short: events", sum(len(t["ts"]) for t in traces))
    _check_set(lib, "diverse", w.trace_cfg(), traces, prof, sc)


def test_stress_32_models_short(lib):
    w = tg.standard(4).scaled(duration_ms=600_000, n_traces=4, proc_params={
        "flash_mult": 10.0, "flash_len_s": 30.0, "flash_first_s": 100.0, "flash_every_s": 200.0,
        "flash_models": 4})
    traces, prof, _ = _workload_set(w, 0, 4)
    sc = _random_scenarios(4, 16, 4)
    say("stress-short: events", sum(len(t["ts"]) for t in traces))
    _check_set(lib, "stress", w.trace_cfg(), traces, prof, sc)


def test_sweep_mixed_scenario_counts(lib):
    """A sweep where traces carry one scenario (replayed inside the stream),
    several (replayed by the separate kernel from the tick snapshot) or none,
    in a shuffled scenario table: every scenario equal to the oracle."""
    w = tg.standard(4).scaled(duration_ms=600_000, n_traces=5, proc_params={
        "flash_mult": 10.0, "flash_len_s": 30.0, "flash_first_s": 100.0, "flash_every_s": 200.0,
        "flash_models": 4})
    traces, prof, _ = _workload_set(w, 0, 5)
    sc = _random_scenarios(5, 7, 44)
    sc["trace"] = np.array([1, 0, 3, 1, 4, 1, 3], np.uint32)  # trace 2 has none, 0 and 4 one, 1 three, 3 two
    say("mixed: events", sum(len(t["ts"]) for t in traces))
    _check_set(lib, "mixed", w.trace_cfg(), traces, prof, sc)


# ------------------------------------------------------------- edge cases
def _cfg(M, window_ms, n_windows, fast_w=5, slow_w=10, budget=None):
    return {"window_ms": window_ms, "duration_ms": window_ms * n_windows,
            "fast_period_ms": window_ms * fast_w, "slow_period_ms": window_ms * slow_w,
            "n_models": M, "budget": budget if budget is not None else 2 * M + 3}


def _prof(M, n_traces, seed, theta_lo=20.0, theta_hi=400.0):
    rng = np.random.default_rng(seed)
    n = M * n_traces
    return {"w_p": rng.uniform(0.05, 0.9, n), "w_q": rng.uniform(1.0, 3.0, n),
            "alpha": rng.uniform(0.05, 1.0, n), "theta": rng.uniform(theta_lo, theta_hi, n),
            "tau_crit": rng.uniform(0.2, 0.6, n), "tau_surplus": rng.uniform(1.1, 2.0, n),
            "r_min": rng.integers(0, 2, n).astype(np.int32), "r_init": np.full(n, 2, np.int32)}


def test_edge_mixed_set(lib):
    """Empty traces, late first events, idle gaps longer than the LDS ring,
    boundary-aligned events, a dense window, ties; ragged column ends and an
    offset first trace."""
    M, win, nW = 8, 100, 3000
    traces = [
        E.trace_random(1, M, win * nW, 3000),
        E.trace_empty(),
        E.trace_sparse(2, M, win, nW, gap_windows=700),
        E.trace_boundaries(M, win, nW),
        E.trace_dense_window(M, win, nW, 1234, 60000),
        E.trace_identical_models(M, win, nW),
        E.trace_empty(),
    ]
    cfg = _cfg(M, win, nW)
    prof = _prof(M, len(traces), 7)
    sc = _random_scenarios(len(traces), 3 * len(traces), 8)
    _check_set(lib, "edge", cfg, traces, prof, sc, pad_front=5, pad_back=3)


@pytest.mark.parametrize("M", [1, 3, 17, 33, 64])
def test_model_counts(lib, M):
    win, nW = 250, 2400
    traces = [E.trace_random(10 + M + i, M, win * nW, 400 * M) for i in range(3)]
    cfg = _cfg(M, win, nW, fast_w=4, slow_w=12)
    _check_set(lib, f"M{M}", cfg, traces, _prof(M, 3, M), _random_scenarios(3, 9, M))


@pytest.mark.parametrize("win,fast_w,slow_w", [(1, 1000, 3000), (7, 3, 5), (1000, 1, 1), (60000, 1, 2)])
def test_window_shapes(lib, win, fast_w, slow_w):
    M = 5
    nW = max(8, min(20000, 3_600_000 // win))
    traces = [E.trace_random(20 + i, M, win * nW, 3000) for i in range(2)]
    cfg = _cfg(M, win, nW, fast_w=fast_w, slow_w=slow_w)
    _check_set(lib, f"win{win}", cfg, traces, _prof(M, 2, win), _random_scenarios(2, 6, win))


def test_idle_budget_and_floors(lib):
    M, win, nW = 6, 500, 4000
    traces = [E.trace_random(30 + i, M, win * nW, 6000, model_weights=[0.5, 0.3, 0.1, 0.05, 0.05, 0.0])
              for i in range(2)]
    cfg = _cfg(M, win, nW, budget=40)
    prof = _prof(M, 2, 9, theta_lo=200.0, theta_hi=2000.0)
    prof["r_min"] = np.array([0, 1, 2, 1, 0, 3] * 2, np.int32)
    prof["r_init"] = np.array([1, 2, 3, 4, 1, 5] * 2, np.int32)
    _check_set(lib, "idlebudget", cfg, traces, prof, _random_scenarios(2, 8, 10))


# ------------------------------------------------------------ determinism
def test_deterministic_across_launches(lib):
    tre, device, torch = lib
    w = tg.standard(4).scaled(duration_ms=300_000, n_traces=3)
    dt = device.upload(w)
    ev = device.load(dt)
    prof = device.profiles(w)
    a = tre.tss_outputs(ev, which=("tss64", "a_int"))
    b = tre.tss_outputs(ev, which=("tss64", "a_int"))
    tre.tre_eval_tss(ev, prof, a)
    tre.tre_eval_tss(ev, prof, b)
    torch.cuda.synchronize()
    assert torch.equal(a["tss64"].view(torch.int64), b["tss64"].view(torch.int64))
    assert torch.equal(a["a_int"], b["a_int"])


# ------------------------------------------------------------- validation
def test_validation_errors(lib):
    tre, device, torch = lib
    M, win, nW = 4, 100, 100
    cfg = _cfg(M, win, nW)
    base = E.trace_random(40, M, win * nW, 300)

    def load(tr, **kw):
        cols, off = _columns_from_host(torch, [tr])
        return tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off,
                                   kw.get("cfg", cfg))

    ev = load(base)
    ev.close()
    bad = {k: v.copy() for k, v in base.items()}
    bad["ts"][10], bad["ts"][11] = bad["ts"][11] + 1, bad["ts"][10]
    with pytest.raises(tre.TreError) as e:
        load(bad)
    assert e.value.code == tre.TRE_EORDER
    bad = {k: v.copy() for k, v in base.items()}
    bad["ts"][-1] = win * nW
    with pytest.raises(tre.TreError) as e:
        load(bad)
    assert e.value.code == tre.TRE_EORDER
    bad = {k: v.copy() for k, v in base.items()}
    bad["model"][5] = M
    with pytest.raises(tre.TreError) as e:
        load(bad)
    assert e.value.code == tre.TRE_ESCHEMA
    bad = {k: v.copy() for k, v in base.items()}
    bad["type"][5] = 0x84
    with pytest.raises(tre.TreError) as e:
        load(bad)
    assert e.value.code == tre.TRE_ESCHEMA
    bad = {k: v.copy() for k, v in base.items()}
    bad["type"][5] = 0x82  # ADMIT on a DECODE
    with pytest.raises(tre.TreError) as e:
        load(bad)
    assert e.value.code == tre.TRE_ESCHEMA
    dense = E.trace_dense_window(M, win, nW, 5, 66000)
    with pytest.raises(tre.TreError) as e:
        load(dense)
    assert e.value.code == tre.TRE_ERANGE
    for c in ({**cfg, "duration_ms": win * nW + 1}, {**cfg, "n_models": 65}, {**cfg, "fast_period_ms": 150}):
        with pytest.raises(tre.TreError) as e:
            load(base, cfg=c)
        assert e.value.code == tre.TRE_EINVAL
    # misaligned column
    cols, off = _columns_from_host(torch, [base])
    with pytest.raises(tre.TreError) as e:
        tre.tre_load_events(cols["ts"][1:], cols["model"], cols["req"], cols["type"], cols["tokens"], off - 1, cfg)
    assert e.value.code == tre.TRE_EINVAL
    # parameter tables
    ev = load(base)
    prof = _prof(M, 1, 1)
    good = tre.pack(prof, tre.PROFILE_DTYPE)
    tre.tre_check_params(ev, good)
    for k, v in (("alpha", 0.0), ("theta", -1.0), ("tau_crit", 3.0)):
        p2 = {kk: vv.copy() for kk, vv in prof.items()}
        p2[k][0] = v
        with pytest.raises(tre.TreError) as e:
            tre.tre_check_params(ev, tre.pack(p2, tre.PROFILE_DTYPE))
        assert e.value.code == tre.TRE_EINVAL
    p2 = {kk: vv.copy() for kk, vv in prof.items()}
    p2["r_init"][:] = 100
    with pytest.raises(tre.TreError):
        tre.tre_check_params(ev, tre.pack(p2, tre.PROFILE_DTYPE))
    sc = _random_scenarios(1, 2, 1)
    sc["trace"][1] = 5
    with pytest.raises(tre.TreError):
        tre.tre_check_params(ev, good, tre.pack(sc, tre.SCENARIO_DTYPE))
    # workspace too small
    sc = tre.pack(_random_scenarios(1, 2, 1), tre.SCENARIO_DTYPE)
    out = tre.ctl_outputs(ev, 2, 10)
    ws = torch.empty(8, dtype=torch.uint8, device="cuda")
    with pytest.raises(tre.TreError) as e:
        tre.tre_sweep(ev, good, sc, out, ws)
    assert e.value.code == tre.TRE_ENOMEM
    ev.close()


def _perturbed(rng, tr, how, duration_ms=None):
    """A copy of a host trace with one change: 'shuffle' permutes the rows
    of every instant (a valid stream stays valid), 'drop_arrive' /
    'drop_admit' delete one row of that kind, 'dup_admit' / 'dup_arrive' /
    'dup_finish' repeat one row of that kind (the same request id) at a
    later row of its instant or after it, 'decode_after' adds a DECODE of a
    finished request one ms after its FINISH, 'decode_same' one listed right
    after its FINISH in the same instant (allowed)."""
    t = {k: v.copy() for k, v in tr.items()}
    n = len(t["ts"])
    if how == "shuffle":
        order = np.lexsort((rng.random(n), t["ts"]))
        return {k: v[order] for k, v in t.items()}
    if how in ("decode_after", "decode_same"):
        fin = np.flatnonzero(t["type"] == 3)
        if how == "decode_after":
            fin = fin[t["ts"][fin] + 1 < duration_ms]
        r = int(rng.choice(fin))
        row = {k: v[r] for k, v in t.items()}
        row["type"] = 2
        row["tokens"] = 5
        if how == "decode_same":
            j = r + 1
        else:
            row["ts"] = int(t["ts"][r]) + 1
            j = int(np.searchsorted(t["ts"], row["ts"]))
        return {k: np.insert(v, j, row[k]) for k, v in t.items()}
    kind = {"drop_arrive": 0, "drop_admit": 0x81, "dup_admit": 0x81, "dup_arrive": 0, "dup_finish": 3}[how]
    rows = np.flatnonzero(t["type"] == kind)
    r = int(rng.choice(rows))
    if how.startswith("drop"):
        keep = np.ones(n, bool)
        keep[r] = False
        return {k: v[keep] for k, v in t.items()}
    j = int(rng.integers(r + 1, n + 1))  # insert a copy of row r before row j (ts kept sorted)
    row = {k: v[r] for k, v in t.items()}
    row["ts"] = max(int(t["ts"][r]), int(t["ts"][j - 1]))
    return {k: np.insert(v, j, row[k]) for k, v in t.items()}


def test_state_validation(lib):
    """TRE_ESTATE at load against the oracle: the active / waiting counts of
    Eq. (1) never below zero at any instant, no request id admitted twice,
    and every id on one lifecycle (one ARRIVE, one FINISH, no ARRIVE or
    DECODE after the FINISH). Traces with many rows per millisecond (so
    instants span the kernel's 64-row steps), perturbed at random: rows of
    one instant shuffled (accepted, same tallies), an ARRIVE or an ADMIT
    dropped, an ADMIT, ARRIVE or FINISH repeated, a DECODE after a FINISH or
    listed after it in the same instant (accepted). The GPU must reject
    exactly what the oracle rejects."""
    tre, device, torch = lib
    o = O.get()
    M, win, nW = 5, 10, 50
    cfg = _cfg(M, win, nW, fast_w=2, slow_w=4)
    rng = np.random.default_rng(77)
    seen = {"ok": 0, "state": 0}
    kinds = ("shuffle", "drop_arrive", "drop_admit", "dup_admit", "dup_arrive", "dup_finish", "decode_after",
             "decode_same")
    for case in range(64):
        how = kinds[case % 8]
        # every request admitted and finished in half the cases, so the
        # counts return to zero and a dropped row takes one below it
        full = (case // 8) % 2 == 1
        base = E.trace_random(500 + case, M, win * nW, 400, max_span_ms=300,
                              **({"admit_p": 1.0, "finish_p": 1.0} if full else {}))
        tr = _perturbed(rng, base, how, win * nW)
        assert (np.diff(tr["ts"]) >= 0).all()
        exp_state = o.trace_status(tr, win, win * nW, M)
        assert exp_state in (0, -5), exp_state
        exp_dup = o.check_admits(tr)[0]
        exp_life = o.check_lifecycle(tr)[0]
        if how in ("dup_arrive", "dup_finish", "decode_after"):
            assert exp_life == -7, how
        if how == "decode_same":
            assert exp_life == 0
        cols, off = _columns_from_host(torch, [tr])
        say(f"state case {case} ({how}): {len(tr['ts'])} rows, oracle {exp_state} / {exp_dup} / {exp_life}")
        if exp_state or exp_dup or exp_life:
            with pytest.raises(tre.TreError) as e:
                tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
            assert e.value.code == tre.TRE_ESTATE, (case, how, str(e.value))
            seen["state"] += 1
        else:
            ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
            if how == "shuffle":
                prof_cols = _prof(M, 1, case)
                prof = tre.pack(prof_cols, tre.PROFILE_DTYPE)
                g = _eval_all(tre, ev, prof)

                class W:
                    window_ms = win
                    duration_ms = win * nW
                ref = PT.oracle_tss(tr, W, PT.trace_profile(prof_cols, 0, M))
                PT.compare_tss({k: v[0] for k, v in g.items()}, ref, f"shuffled instants, case {case}")
            ev.close()
            seen["ok"] += 1
        # the same columns without request ids: only the counts are checked
        if (exp_dup or exp_life) and not exp_state:
            ev = tre.tre_load_events(cols["ts"], cols["model"], None, cols["type"], cols["tokens"], off, cfg)
            ev.close()
    say("state validation:", seen)
    assert seen["ok"] >= 20 and seen["state"] >= 30


def test_lifecycle_validation_across_traces(lib):
    """The lifecycle check over several traces at once, with sparse large
    request ids (per-trace tables sized by the largest ARRIVE or FINISH
    id): accepted when every trace is valid; otherwise TRE_ESTATE naming the
    smallest trace in error, whichever trace holds it."""
    tre, device, torch = lib
    o = O.get()
    M, win, nW = 3, 100, 20
    cfg = _cfg(M, win, nW, fast_w=2, slow_w=4)
    ARR, ADM, DEC, FIN = 0, 0x81, 2, 3

    def life(rid, m, t0, t1):
        return [(t0, m, rid, ARR, 5), (t0, m, rid, ADM, 5), (t1, m, rid, DEC, 3), (t1, m, rid, FIN, 0)]

    def tr(rows):
        return E._pack(rows)

    good = [tr(life(7, 0, 10, 500) + life(3_000_000, 1, 20, 700)),
            tr(life(1, 2, 5, 1999) + life(999_999, 0, 100, 1500) + [(1500, 0, 999_999, DEC, 2)]),
            tr(life(42, 1, 0, 10))]
    for t in good:
        assert o.check_lifecycle(t) == (0, None)
    cols, off = _columns_from_host(torch, good)
    tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg).close()
    for bad_at in (0, 1, 2):
        traces = [dict(t) for t in good]
        rows = life(2_000_000 + bad_at, 0, 30, 600) + [(601, 0, 2_000_000 + bad_at, DEC, 1)]
        traces[bad_at] = tr(rows + life(5, 1, 40, 50))
        assert o.check_lifecycle(traces[bad_at]) == (-7, 2_000_000 + bad_at)
        cols, off = _columns_from_host(torch, traces)
        with pytest.raises(tre.TreError) as e:
            tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
        assert e.value.code == tre.TRE_ESTATE and f"trace {bad_at}:" in str(e.value), str(e.value)


def test_state_validation_hand_cases(lib):
    """Hand-built streams at chunk-boundary positions: a FINISH with nothing
    active, an ADMIT with nothing waiting and a second ADMIT of one id, each
    placed so that the failing instant is inside a 64-row step, at its last
    row, across two steps, or at the last row of the trace; and an instant
    out of lifecycle order straddling two steps (accepted)."""
    tre, device, torch = lib
    o = O.get()
    M, win, nW = 3, 1000, 4
    cfg = _cfg(M, win, nW, fast_w=1, slow_w=2)
    ARR, ADM, DEC, FIN = 0, 0x81, 2, 3

    def filler(n, t0=0):  # n complete requests of model 2, one row per ms from t0
        rows = []
        for r in range(n // 4):
            t = t0 + 4 * r
            rows += [(t, 2, 1000 + r, ARR, 3), (t + 1, 2, 1000 + r, ADM, 3), (t + 2, 2, 1000 + r, DEC, 2),
                     (t + 3, 2, 1000 + r, FIN, 0)]
        return rows

    def run(rows, expect_state):
        tr = E._pack(rows)
        assert o.trace_status(tr, win, win * nW, M) == (-5 if expect_state == "count" else 0)
        assert o.check_admits(tr)[0] == (-6 if expect_state == "dup" else 0)
        cols, off = _columns_from_host(torch, [tr])
        if expect_state:
            with pytest.raises(tre.TreError) as e:
                tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
            assert e.value.code == tre.TRE_ESTATE, str(e.value)
        else:
            tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg).close()

    for lead in (0, 60, 62, 63, 64, 124, 127):
        f = filler(lead)
        t = 4 * (lead // 4) + 10
        # FINISH with nothing active (model 0), then its ADMIT at a later instant
        run(f + [(t, 0, 1, ARR, 5), (t + 1, 0, 1, FIN, 0), (t + 2, 0, 1, ADM, 5)], "count")
        # ADMIT with nothing waiting (model 1)
        run(f + [(t, 1, 2, ADM, 5), (t + 1, 1, 2, FIN, 0)], "count")
        # the same rows at one instant, ADMIT first: accepted
        run(f + [(t, 1, 2, ADM, 5), (t, 1, 2, ARR, 5), (t + 1, 1, 2, FIN, 0)], None)
        # an instant of 70 rows, out of lifecycle order, crossing a step
        burst = [(t, 0, 10 + k, ADM, 1) for k in range(35)] + [(t, 0, 10 + k, ARR, 1) for k in range(35)]
        run(f + burst, None)
        # the same with one ARRIVE short: negative after the instant
        run(f + burst[:-1], "count")
        # a second ADMIT of one id (another request keeps the waiting count up)
        run(f + [(t, 0, 5, ARR, 5), (t, 0, 6, ARR, 5), (t + 1, 0, 5, ADM, 5), (t + 2, 0, 5, ADM, 5)], "dup")
        # negative at the very last row of the trace
        run(f + [(t, 1, 3, ARR, 5), (t + 1, 1, 3, ADM, 5), (3999, 1, 3, FIN, 0), (3999, 1, 3, FIN, 0)], "count")


def test_validation_reports_lowest_row_kind(lib):
    """The message names the kind of the lowest failing row: a schema error
    at row 5 with an unsorted timestamp at row 50 is TRE_ESCHEMA at row 5,
    and the other way round TRE_EORDER."""
    tre, device, torch = lib
    M, win, nW = 4, 100, 100
    cfg = _cfg(M, win, nW)
    base = E.trace_random(40, M, win * nW, 300)

    def load(tr):
        cols, off = _columns_from_host(torch, [tr])
        return tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)

    bad = {k: v.copy() for k, v in base.items()}
    bad["model"][5] = M
    bad["ts"][50], bad["ts"][51] = bad["ts"][51] + 1, bad["ts"][50]
    with pytest.raises(tre.TreError) as e:
        load(bad)
    assert e.value.code == tre.TRE_ESCHEMA and "row 5:" in str(e.value), str(e.value)
    assert O.get().trace_status(bad, win, win * nW, M) == -3
    bad = {k: v.copy() for k, v in base.items()}
    bad["model"][50] = M
    bad["ts"][5], bad["ts"][6] = bad["ts"][6] + 1, bad["ts"][5]
    with pytest.raises(tre.TreError) as e:
        load(bad)
    assert e.value.code == tre.TRE_EORDER and "row 6:" in str(e.value), str(e.value)
    assert O.get().trace_status(bad, win, win * nW, M) == -2


def test_move_log_capacity(lib):
    """A short move log keeps the first entries; n_moves still counts all."""
    tre, device, torch = lib
    w = tg.standard(2)
    traces, prof_cols, _ = _workload_set(w, 0, 1)
    sc_cols = w.scenario_columns()
    sc_cols = {k: v[:64] for k, v in sc_cols.items()}
    cols, off = _columns_from_host(torch, traces)
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, w.trace_cfg())
    prof = tre.pack(prof_cols, tre.PROFILE_DTYPE)
    sc = tre.pack(sc_cols, tre.SCENARIO_DTYPE)
    ws = torch.empty(tre.tre_workspace_size(ev, 64), dtype=torch.uint8, device="cuda")
    big = tre.ctl_outputs(ev, 64, ev.n_ticks * 4)
    small = tre.ctl_outputs(ev, 64, 3)
    tre.tre_sweep(ev, prof, sc, big, ws)
    tre.tre_sweep(ev, prof, sc, small, ws)
    mb = tre.unpack_moves(big["moves"]).reshape(64, -1)
    ms = tre.unpack_moves(small["moves"]).reshape(64, -1)
    assert torch.equal(big["n_moves"], small["n_moves"])
    for s in range(64):
        k = min(3, int(big["n_moves"][s]))
        assert np.array_equal(mb[s, :k], ms[s, :k])
    assert int(big["n_moves"].max()) > 3
    ev.close()
