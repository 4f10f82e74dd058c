"""Pins of the closed-loop replay oracle (oracle/tre_oracle_loop.c).

Each pin takes an ``oracle.Oracle`` and raises AssertionError when the
oracle disagrees with something fixed independently of it:
- with no moves allowed, its events and latency outcomes equal an
  independent open-loop simulation (one heap of slot free times per model);
- its move log, final replicas and replica-window sums equal the base
  control replay (itself pinned) run over the closed loop's own final TSS;
- a hand-derived case where a rescue adds a replica at a window end, the
  replica cap blocks a receiver, and a donor's slot leaves;
- conservation (arrived / started / judged requests against the events);
- more initial replicas never delay a request (FCFS on more servers);
- with the actuation model: no delays, unit footprints and no vetoes give
  the plain closed loop; the move log, replicas, replica-window sums and
  GPU accounting equal the actuation replay (tre_oracle_act.c, itself
  pinned) run over the closed loop's own final TSS; a hand-derived case
  where the wake and sleep delays decide when a waiting request starts;
  GPU conservation, no vetoed donor and at most K moves per tick.

Readings followed (paper, Sections "Dual-Speed Control", "Bounded Pairwise
Transfer", "System Boundary and Replica State"): FCFS per model on the slot
that frees first, whole-millisecond service per chunk, a move acting from
the end of its window, a donor's earliest-free slots leaving.
"""
import heapq
import math

import numpy as np

import oracle as O
import tracegen as tg

A, P, D, F, ADMIT = 0, 1, 2, 3, 0x80
RES, POOL = 1, 0xFF


def _sc(K, theta_scale=1.0, tau=-1.0):
    sc = np.zeros(1, O.SCENARIO_DTYPE)
    sc["max_moves"], sc["theta_scale"], sc["tau_crit_override"] = K, theta_scale, tau
    return sc


def _open_loop(reqs, M, svc, slo, slots, dur, pchunk=2048, dchunk=24):
    """Independent statement of FCFS service on a fixed number of slots."""
    events = []
    stats = {m: [0, 0, 0, 0] for m in range(M)}  # n_done, n_ok, e2e_sum, e2e_max
    for m in range(M):
        sel = np.nonzero(reqs["model"] == m)[0]
        heap = [0] * slots[m]
        for i in sel:
            a, p, o = int(reqs["arrival_ms"][i]), int(reqs["prompt"][i]), int(reqs["output"][i])
            events.append((a, m, A, p))
            if not heap:
                continue
            s = max(a, heapq.heappop(heap))
            t, left, first = s, p, True
            while left > 0:
                ch = min(left, pchunk)
                events.append((t, m, P | (ADMIT if first else 0), ch))
                first = False
                t += -(-ch * int(svc[m]["prefill_us"]) // 1000)
                left -= ch
            left, t_first, first_ch = o, None, 0
            while left > 0:
                ch = min(left, dchunk)
                t += -(-ch * int(svc[m]["decode_us"]) // 1000)
                if t_first is None:
                    t_first, first_ch = t, ch
                events.append((t, m, D, ch))
                left -= ch
            events.append((t, m, F, 0))
            heapq.heappush(heap, t)
            if t < dur:
                ttft, e2e = t_first - a, t - a
                good = ttft <= slo[m]["ttft_ms"] and e2e <= slo[m]["e2e_ms"]
                if o - first_ch > 0:
                    good = good and (t - t_first) / (o - first_ch) <= slo[m]["tpot_ms"]
                st = stats[m]
                st[0] += 1; st[1] += int(good); st[2] += e2e; st[3] = max(st[3], e2e)
    events = sorted(e for e in events if e[0] < dur)
    return events, stats


def _workloads():
    out = []
    w = tg.standard(0)
    out.append((w, w.requests(0)))
    w = tg.standard(1).scaled(duration_ms=600_000)
    out.append((w, w.requests(0)))
    return out


def _inputs(w):
    prof = O.pack_profiles(w.profile_columns(1))
    return prof, O.pack_slo(w.slo_columns(1)), O.pack_svc(w.service_columns(1))


def pin_without_moves_equals_open_loop_service(o):
    for w, reqs in _workloads():
        prof, slo, svc = _inputs(w)
        for extra in (0, 1):  # the workload's slots, and one replica more per model
            prof2 = prof.copy()
            prof2["r_init"] += extra
            cfg = dict(w.trace_cfg(), budget=int(prof2["r_init"].sum()))
            r = o.loop(cfg, prof2, _sc(0), slo, svc, reqs, want_events=True)
            got = sorted(zip(r["events"]["ts"].tolist(), r["events"]["model"].tolist(),
                             r["events"]["type"].tolist(), r["events"]["tokens"].tolist()))
            exp, st = _open_loop(reqs, w.n_models, svc, slo, [8 * int(x) for x in prof2["r_init"]], w.duration_ms)
            assert got == exp, (w.name, extra)
            for m in range(w.n_models):
                s = r["stats"][m]
                assert [int(s["n_done"]), int(s["n_ok"]), int(s["e2e_sum"]), int(s["e2e_max"])] == st[m], (w.name, m)
            assert r["n_moves"] == 0 and np.array_equal(r["r_final"], prof2["r_init"])


def pin_moves_equal_the_base_replay_over_the_loops_own_tss(o):
    rng = np.random.default_rng(21)
    for w, reqs in _workloads():
        prof, slo, svc = _inputs(w)
        for it in range(8):
            sc = _sc(int(rng.choice([1, 2, 4])), float(rng.uniform(0.5, 2.0)),
                     float(rng.choice([-1.0, rng.uniform(0.2, 0.8)])))
            cfg = dict(w.trace_cfg(), budget=int(prof["r_init"].sum()) + int(rng.integers(0, 4)))
            r = o.loop(cfg, prof, sc, slo, svc, reqs, r_cap=10_000, want_tss=True)
            base = o.control(cfg, prof, r["S"], r["flags"], sc)
            assert r["n_moves"] == base["n_moves"], (w.name, it)
            assert np.array_equal(r["moves"], base["moves"]), (w.name, it)
            assert np.array_equal(r["r_final"], base["r_final"]) and np.array_equal(r["r_windows"], base["r_windows"])
            if it == 0:
                assert r["n_moves"] > 0, "the workload should see some moves"


def _hand(o, r_cap):
    # M = 2, one slot per replica, 1 replica each, budget 3 (one idle GPU),
    # windows of 100 ms, every window a fast and slow tick. Model 0: three
    # requests at t = 0, prompt 1 token (1 ms), output 24 tokens (one chunk,
    # 240 ms); model 1 has none (idle: a surplus donor). theta is huge, so a
    # non-idle model 0 is critical at every tick.
    #  w0: r0 starts at 0 (PREFILL 0, DECODE / FINISH 241); r1, r2 wait.
    #  tick 0: rescue, idle GPU -> model 0 gains a slot free at 100.
    #  w1: r1 starts at 100 (FINISH 341); r2 needs a slot before 200: none.
    #  tick 1: rescue again. r_cap 3: donor model 1 (idle, R 1 > floor 0)
    #    -> model 0 gains a slot free at 200; r_cap 2: no receiver.
    #  w2: r2 starts at 200 (FINISH 441) with r_cap 3; with r_cap 2 at 241
    #    when r0's slot frees (FINISH 482).
    cfg = {"window_ms": 100, "duration_ms": 1000, "fast_period_ms": 100, "slow_period_ms": 100,
           "n_models": 2, "budget": 3}
    prof = np.zeros(2, O.PROFILE_DTYPE)
    prof["w_p"], prof["w_q"], prof["alpha"], prof["theta"] = 0.5, 2.0, 1.0, 1e12
    prof["tau_crit"], prof["tau_surplus"], prof["r_min"], prof["r_init"] = 0.5, 1.5, 0, 1
    slo = np.zeros(2, O.SLO_DTYPE)
    slo["ttft_ms"] = slo["tpot_ms"] = slo["e2e_ms"] = 1e9
    svc = np.zeros(2, O.SVC_DTYPE)
    svc["prefill_us"], svc["decode_us"] = 1000, 10000
    reqs = {"arrival_ms": np.zeros(3, np.int64), "model": np.zeros(3, np.uint8), "prompt": np.ones(3, np.uint16),
            "output": np.full(3, 24, np.uint16)}
    return o.loop(cfg, prof, _sc(1), slo, svc, reqs, spr=1, r_cap=r_cap, want_events=True)


def pin_hand_rescue_cap_and_donor(o):
    r = _hand(o, 3)
    mv = [(int(m["window"]), int(m["path"]), int(m["receiver"]), int(m["donor"])) for m in r["moves"]]
    assert mv[:2] == [(0, RES, 0, POOL), (1, RES, 0, 1)], mv
    ev = r["events"]
    fin = sorted(int(t) for t, ty in zip(ev["ts"], ev["type"]) if ty == F)
    adm = sorted(int(t) for t, ty in zip(ev["ts"], ev["type"]) if ty == (P | ADMIT))
    assert adm == [0, 100, 200] and fin == [241, 341, 441], (adm, fin)
    s = r["stats"][0]
    assert (int(s["n_done"]), int(s["e2e_sum"]), int(s["e2e_max"])) == (3, 241 + 341 + 441, 441)
    r = _hand(o, 2)
    mv = [(int(m["window"]), int(m["path"]), int(m["receiver"]), int(m["donor"])) for m in r["moves"]]
    assert mv == [(0, RES, 0, POOL)], mv  # model 0 at its cap from then on
    ev = r["events"]
    adm = sorted(int(t) for t, ty in zip(ev["ts"], ev["type"]) if ty == (P | ADMIT))
    assert adm == [0, 100, 241]
    assert int(r["stats"][0]["e2e_max"]) == 482 and list(r["r_final"]) == [2, 1]


def pin_donor_releases_its_earliest_free_slots(o):
    # M = 2, two slots per replica, budget 3 (no idle GPU). Model 0: one
    # replica, theta huge (critical while active), r_cap 2; three requests at
    # t = 0 (prompt 1, output 24: 241 ms each). Model 1: two replicas (four
    # slots), theta tiny (surplus), requests at t = 0 with outputs 48 and 72
    # (FINISH at 481 and 721) and one at t = 150 (output 24).
    #  w0: model 0 starts two (slots free at 241), the third waits; model 1
    #      starts its two (slots at 481 and 721, two slots idle).
    #  tick 0: rescue, donor model 1: its two earliest-free slots (the idle
    #      ones) leave; model 0 gains two slots free at 100.
    #  w1: model 0's third request starts at 100 (FINISH 341).
    #  model 1's request at 150 waits for the slot freeing at 481.
    #  Model 1 is also critical in windows with requests but no tokens
    #  (TSS 0, alpha 1): at ticks 1 and 3 its donor would be model 0, still
    #  critical itself (active until 341), so no move; at tick 5 model 0 is
    #  idle (a surplus donor) and model 1 (1 replica, below r_cap) receives
    #  a replica from it.
    cfg = {"window_ms": 100, "duration_ms": 2000, "fast_period_ms": 100, "slow_period_ms": 100,
           "n_models": 2, "budget": 3}
    prof = np.zeros(2, O.PROFILE_DTYPE)
    prof["w_p"], prof["w_q"], prof["alpha"] = 0.5, 2.0, 1.0
    prof["theta"] = [1e12, 1e-12]
    prof["tau_crit"], prof["tau_surplus"], prof["r_min"], prof["r_init"] = 0.5, 1.5, 0, [1, 2]
    slo = np.zeros(2, O.SLO_DTYPE)
    slo["ttft_ms"] = slo["tpot_ms"] = slo["e2e_ms"] = 1e9
    svc = np.zeros(2, O.SVC_DTYPE)
    svc["prefill_us"], svc["decode_us"] = 1000, 10000
    reqs = {"arrival_ms": np.array([0, 0, 0, 0, 0, 150], np.int64), "model": np.array([0, 0, 0, 1, 1, 1], np.uint8),
            "prompt": np.ones(6, np.uint16), "output": np.array([24, 24, 24, 48, 72, 24], np.uint16)}
    r = o.loop(cfg, prof, _sc(1), slo, svc, reqs, spr=2, r_cap=2, want_events=True)
    mv = [(int(m["window"]), int(m["path"]), int(m["receiver"]), int(m["donor"])) for m in r["moves"]]
    assert mv == [(0, RES, 0, 1), (5, RES, 1, 0)], mv
    ev = r["events"]
    adm = {m: sorted(int(t) for t, mm, ty in zip(ev["ts"], ev["model"], ev["type"]) if ty == (P | ADMIT) and mm == m)
           for m in (0, 1)}
    assert adm == {0: [0, 0, 100], 1: [0, 0, 481]}, adm
    assert list(r["r_final"]) == [1, 2]


def pin_conservation(o):
    for w, reqs in _workloads():
        prof, slo, svc = _inputs(w)
        cfg = dict(w.trace_cfg(), budget=int(prof["r_init"].sum()) + 2)
        r = o.loop(cfg, prof, _sc(2), slo, svc, reqs, want_events=True)
        ev = r["events"]
        assert (np.diff(ev["ts"]) >= 0).all() and (ev["ts"] < w.duration_ms).all()
        for m in range(w.n_models):
            s = r["stats"][m]
            sel = ev["model"] == m
            assert int(s["n_arrived"]) == int(np.sum(reqs["model"] == m)) == int(np.sum(sel & (ev["type"] == A)))
            assert int(s["n_started"]) == int(np.sum(sel & (ev["type"] == (P | ADMIT))))
            assert int(s["n_done"]) == int(np.sum(sel & (ev["type"] == F)))
            assert int(s["n_ok"]) <= int(s["n_done"]) <= int(s["n_started"]) <= int(s["n_arrived"])
        # replicas: budget conservation at the end
        assert int(r["r_final"].sum()) <= cfg["budget"]


def pin_more_replicas_never_delay(o):
    for w, reqs in _workloads():
        prof, slo, svc = _inputs(w)
        prev = None
        for extra in (0, 1, 3):
            p2 = prof.copy()
            p2["r_init"] += extra
            cfg = dict(w.trace_cfg(), budget=int(p2["r_init"].sum()))
            r = o.loop(cfg, p2, _sc(0), slo, svc, reqs)
            cur = r["stats"]
            if prev is not None:
                assert (cur["n_done"] >= prev["n_done"]).all()
                assert (cur["n_started"] >= prev["n_started"]).all()
            prev = cur


def pin_bad_arguments_are_rejected(o):
    w, reqs = _workloads()[0]
    prof, slo, svc = _inputs(w)
    cfg = w.trace_cfg()
    for kw, c in (({"spr": 0}, cfg), ({"r_cap": 1}, cfg), ({}, dict(cfg, budget=1))):
        try:
            o.loop(c, prof, _sc(1), slo, svc, reqs, **kw)
        except ValueError:
            continue
        raise AssertionError(f"accepted {kw} {c['budget']}")


def _act_inputs(rng, w, nW_ticks):
    M = w.n_models
    g = rng.integers(1, 3, M).astype(np.int32)
    veto = rng.integers(0, 1 << 62, nW_ticks, dtype=np.int64).astype(np.uint64) & np.uint64((1 << M) - 1)
    veto[rng.random(nW_ticks) > 0.2] = 0
    return g, veto


def _n_ticks(cfg):
    nW = cfg["duration_ms"] // cfg["window_ms"]
    return sum(1 for x in range(nW) if ((x + 1) * cfg["window_ms"]) % cfg["fast_period_ms"] == 0
               or ((x + 1) * cfg["window_ms"]) % cfg["slow_period_ms"] == 0)


def pin_act_without_delays_is_the_plain_loop(o):
    rng = np.random.default_rng(31)
    for w, reqs in _workloads():
        prof, slo, svc = _inputs(w)
        for it in range(3):
            sc = _sc(int(rng.choice([1, 2, 4])), float(rng.uniform(0.5, 2.0)))
            cfg = dict(w.trace_cfg(), budget=int(prof["r_init"].sum()) + int(rng.integers(0, 4)))
            a = o.loop(cfg, prof, sc, slo, svc, reqs, want_tss=True)
            b = o.loop(cfg, prof, sc, slo, svc, reqs, want_tss=True, wake_w=0, sleep_w=0,
                       footprint=np.ones(w.n_models, np.int32), veto=np.zeros(_n_ticks(cfg), np.uint64))
            assert a["n_moves"] == b["n_moves"] and np.array_equal(a["moves"], b["moves"]), (w.name, it)
            for k in ("r_final", "r_windows", "stats", "flags"):
                assert np.array_equal(a[k], b[k]), (w.name, it, k)
            assert np.array_equal(a["S"].view(np.uint64), b["S"].view(np.uint64)), (w.name, it)
            assert b["idle_final"] == cfg["budget"] - int(b["r_final"].sum()) and not b["held_final"].any()


def pin_act_moves_follow_the_actuation_replay(o):
    """The closed loop decides on the TSS of its own service; replaying the
    actuation rules (tre_oracle_act.c) over that TSS must give its moves."""
    rng = np.random.default_rng(33)
    for w, reqs in _workloads():
        prof, slo, svc = _inputs(w)
        total = 0
        for it, (wake_w, sleep_w) in enumerate([(2, 3), (0, 4), (5, 0), (1, 1)]):
            cfg = dict(w.trace_cfg())
            g, veto = _act_inputs(rng, w, _n_ticks(cfg))
            cfg["budget"] = int((g * prof["r_init"]).sum()) + int(rng.integers(0, 5))
            sc = _sc(int(rng.choice([1, 2, 4])), float(rng.uniform(0.5, 2.0)))
            r = o.loop(cfg, prof, sc, slo, svc, reqs, r_cap=10_000, want_tss=True, wake_w=wake_w, sleep_w=sleep_w,
                       footprint=g, veto=veto)
            a = o.control_act(cfg, prof, r["S"], r["flags"], sc, wake_w, sleep_w, footprint=g, veto=veto)
            assert r["n_moves"] == a["n_moves"] and np.array_equal(r["moves"], a["moves"]), (w.name, it)
            assert np.array_equal(r["r_final"], a["r_final"]) and np.array_equal(r["r_windows"], a["r_windows"])
            assert r["idle_final"] == a["idle_final"] and np.array_equal(r["held_final"], a["held_final"])
            total += r["n_moves"]
        assert total > 0, f"{w.name}: the workload should see some moves"


def pin_act_hand_wake_and_sleep_delays(o):
    # The hand case above with wake_w = 2, sleep_w = 1, r_cap 3:
    #  w0: r0 starts at 0 (FINISH 241); r1, r2 wait.
    #  tick 0: rescue from the idle GPU: model 0's wake runs through
    #    window 2, its slot is free from 300 (window 3).
    #  ticks 1, 2: model 0 critical, but with a wake in flight: no receiver.
    #  w2: r1 starts at 241 on r0's slot (FINISH 482).
    #  w3: the new slot: r2 starts at 300 (FINISH 541).
    #  tick 3: rescue, no idle GPU: donor model 1 (idle: surplus, above its
    #    floor) hidden at once; its sleep runs through window 4, then model
    #    0's wake through window 6: routable from window 7.
    #  r_final [3, 0]; r_windows: model 0 1 x 3 + 2 x 4 + 3 x 3 = 20,
    #  model 1 1 x 4 = 4; no GPU idle or held at the end.
    cfg = {"window_ms": 100, "duration_ms": 1000, "fast_period_ms": 100, "slow_period_ms": 100,
           "n_models": 2, "budget": 3}
    prof = np.zeros(2, O.PROFILE_DTYPE)
    prof["w_p"], prof["w_q"], prof["alpha"], prof["theta"] = 0.5, 2.0, 1.0, 1e12
    prof["tau_crit"], prof["tau_surplus"], prof["r_min"], prof["r_init"] = 0.5, 1.5, 0, 1
    slo = np.zeros(2, O.SLO_DTYPE)
    slo["ttft_ms"] = slo["tpot_ms"] = slo["e2e_ms"] = 1e9
    svc = np.zeros(2, O.SVC_DTYPE)
    svc["prefill_us"], svc["decode_us"] = 1000, 10000
    reqs = {"arrival_ms": np.zeros(3, np.int64), "model": np.zeros(3, np.uint8), "prompt": np.ones(3, np.uint16),
            "output": np.full(3, 24, np.uint16)}
    r = o.loop(cfg, prof, _sc(1), slo, svc, reqs, spr=1, r_cap=3, want_events=True, wake_w=2, sleep_w=1,
               footprint=np.ones(2, np.int32))
    mv = [(int(m["window"]), int(m["path"]), int(m["receiver"]), int(m["donor"])) for m in r["moves"]]
    assert mv == [(0, RES, 0, POOL), (3, RES, 0, 1)], mv
    ev = r["events"]
    adm = sorted(int(t) for t, ty in zip(ev["ts"], ev["type"]) if ty == (P | ADMIT))
    fin = sorted(int(t) for t, ty in zip(ev["ts"], ev["type"]) if ty == F)
    assert adm == [0, 241, 300] and fin == [241, 482, 541], (adm, fin)
    assert list(r["r_final"]) == [3, 0] and list(r["r_windows"]) == [20, 4]
    assert r["idle_final"] == 0 and not r["held_final"].any()


def pin_act_conservation(o):
    rng = np.random.default_rng(35)
    for w, reqs in _workloads():
        prof, slo, svc = _inputs(w)
        cfg = dict(w.trace_cfg())
        nt = _n_ticks(cfg)
        g, veto = _act_inputs(rng, w, nt)
        cfg["budget"] = int((g * prof["r_init"]).sum()) + 3
        K = 4
        r = o.loop(cfg, prof, _sc(K, 1.5), slo, svc, reqs, wake_w=3, sleep_w=2, footprint=g, veto=veto)
        assert r["idle_final"] + int((g * r["r_final"]).sum()) + int(r["held_final"].sum()) == cfg["budget"]
        tick_of = {}
        for x in range(cfg["duration_ms"] // cfg["window_ms"]):
            if ((x + 1) * cfg["window_ms"]) % cfg["fast_period_ms"] == 0 or \
               ((x + 1) * cfg["window_ms"]) % cfg["slow_period_ms"] == 0:
                tick_of[x] = len(tick_of)
        per_tick = {}
        for m in r["moves"]:
            wdw, d = int(m["window"]), int(m["donor"])
            per_tick[wdw] = per_tick.get(wdw, 0) + 1
            if d != POOL:
                assert not (int(veto[tick_of[wdw]]) >> d) & 1, "a vetoed donor released"
        assert max(per_tick.values(), default=0) <= K


ALL = [pin_without_moves_equals_open_loop_service, pin_moves_equal_the_base_replay_over_the_loops_own_tss,
       pin_hand_rescue_cap_and_donor, pin_donor_releases_its_earliest_free_slots, pin_conservation, pin_more_replicas_never_delay, pin_bad_arguments_are_rejected,
       pin_act_without_delays_is_the_plain_loop, pin_act_moves_follow_the_actuation_replay,
       pin_act_hand_wake_and_sleep_delays, pin_act_conservation]
