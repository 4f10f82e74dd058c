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
- more initial replicas never delay a request (FCFS on more servers).

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


ALL = [pin_without_moves_equals_open_loop_service, pin_moves_equal_the_base_replay_over_the_loops_own_tss,
       pin_hand_rescue_cap_and_donor, pin_donor_releases_its_earliest_free_slots, pin_conservation, pin_more_replicas_never_delay, pin_bad_arguments_are_rejected]
