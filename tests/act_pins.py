"""Pins of the actuation-model control replay (oracle/tre_oracle_act.c),
run against the oracle and against planted mistakes.

- Reduction: with instantaneous actuation (no delays, one GPU per replica,
  no vetoes) the replay is the base replay, which the base pins fix.
- Hand-derived cases, each worked out step by step below from the rules in
  the oracle's header: a wake delay and a transfer in flight that blocks a
  later rescue; footprints that make a donor infeasible; the excess GPUs of
  a larger donor returning to the pool when its sleep completes; a vetoed
  donor.
- Invariants on random inputs: GPUs are conserved (idle + sum g * R + held
  by transitions in flight = budget) and no tick makes more than K moves.
"""
import numpy as np

import oracle as O
import tracegen as tg
import edge_traces as E

INIT = 2  # flags: initialised, not idle


def _cfg(M, nW, budget, fast_w=1, slow_w=2):
    return {"window_ms": 1000, "duration_ms": 1000 * nW, "fast_period_ms": 1000 * fast_w,
            "slow_period_ms": 1000 * slow_w, "n_models": M, "budget": budget}


def _prof(r_init, tau_c=0.5, tau_s=1.5, r_min=0):
    M = len(r_init)
    p = np.zeros(M, O.PROFILE_DTYPE)
    p["w_p"], p["w_q"], p["alpha"], p["theta"] = 0.2, 2.0, 0.5, 1.0  # theta = 1: Z = S
    p["tau_crit"], p["tau_surplus"], p["r_min"], p["r_init"] = tau_c, tau_s, r_min, r_init
    return p


def _sc(K=1):
    sc = np.zeros(1, O.SCENARIO_DTYPE)
    sc["max_moves"], sc["theta_scale"], sc["tau_crit_override"] = K, 1.0, -1.0
    return sc


def _const_S(nW, z):
    return np.tile(np.asarray(z, np.float64), (nW, 1)), np.full((nW, len(z)), INIT, np.uint8)


def _moves(r):
    return [(int(m["window"]), int(m["path"]), int(m["receiver"]), int(m["donor"])) for m in r["moves"]]


RES, POOL = O.RESCUE, O.POOL


def pin_wake_delay_blocks_the_receiver_until_routable(o):
    # M = 2, one GPU each, budget 3 (1 idle), model 0 critical (Z 0.2), model 1
    # nominal (Z 1.0), every window a fast tick, K = 1, wake 2 windows.
    #  w0: rescue 0 from the idle GPU, wake until the end of w2 (routable from w3)
    #  w1, w2: 0 is in flight -> no receiver
    #  w3: 0 routable (R0 = 2); rescue 0 again: no idle GPU, donor 1 (nominal,
    #      R 1 > floor 0, Z 1 > 0.2) hidden at once (R1 = 0 from w4), sleep 0
    #      windows, 0 wakes after the sleep: until 3 + 0 + 2 = 5
    #  w4, w5: 0 in flight; w6: 0 routable (R0 = 3), donor 1 at its floor -> none
    # routable per window: (1,1) (1,1) (1,1) (2,1) (2,0) (2,0) (3,0)
    S, f = _const_S(7, [0.2, 1.0])
    r = o.control_act(_cfg(2, 7, 3), _prof([1, 1]), S, f, _sc(1), wake_w=2, sleep_w=0)
    assert _moves(r) == [(0, RES, 0, POOL), (3, RES, 0, 1)]
    assert list(r["r_windows"]) == [12, 4]
    assert list(r["r_final"]) == [3, 0]
    assert r["idle_final"] == 0 and list(r["held_final"]) == [0, 0]


def pin_footprint_feasibility_picks_the_donor_and_blocks_later_moves(o):
    # M = 3, footprints (2, 1, 1), budget 6 with R = (1, 1, 2): 1 idle GPU.
    # Model 0 critical (0.2), models 1, 2 surplus (2.0, 3.0); sleep 1, wake 1.
    #  w0: receiver 0 needs 2 GPUs; 1 idle < 2 -> donors need idle >= 2 - 1:
    #      both feasible, argmax Z -> donor 2; shortfall 1 taken from idle (0);
    #      R2 = 1 from w1; 2 sleeps until w1; 0 wakes until 0 + 1 + 1 = 2
    #  w1, w2: 0 in flight
    #  w3: 0 routable (R0 = 2); receiver 0 again: idle 0 < 2 and no donor has
    #      idle >= 1 -> no move (also w4)
    # routable: (1,1,2) (1,1,1) (1,1,1) (2,1,1) (2,1,1)
    S, f = _const_S(5, [0.2, 2.0, 3.0])
    r = o.control_act(_cfg(3, 5, 6), _prof([1, 1, 2]), S, f, _sc(1), wake_w=1, sleep_w=1,
                            footprint=np.array([2, 1, 1]))
    assert _moves(r) == [(0, RES, 0, 2)]
    assert list(r["r_windows"]) == [7, 5, 6]
    assert list(r["r_final"]) == [2, 1, 1]
    assert r["idle_final"] == 0


def pin_larger_donor_returns_its_excess_after_the_sleep(o):
    # M = 2, footprints (1, 2), budget 3 with R = (1, 1): no idle GPU. Model 0
    # critical, model 1 surplus (2.0); sleep 2, wake 1.
    #  w0: receiver 0 (1 GPU); donor 1 (2 GPUs, feasible): R1 = 0 from w1,
    #      sleep until w2 with 1 GPU to return; 0 wakes until 0 + 2 + 1 = 3
    #  w1, w2: 0 in flight
    #  w3: 1's sleep done -> idle 1; 0 still waking (until 3)
    #  w4: 0 routable (R0 = 2); rescue 0 from the idle GPU: wake until 5
    #  w5: in flight; the wake completes at the end of the last window -> R0 = 3
    # routable: (1,1) (1,0) (1,0) (1,0) (2,0) (2,0)
    S, f = _const_S(6, [0.2, 2.0])
    r = o.control_act(_cfg(2, 6, 3), _prof([1, 1]), S, f, _sc(1), wake_w=1, sleep_w=2,
                            footprint=np.array([1, 2]))
    assert _moves(r) == [(0, RES, 0, 1), (4, RES, 0, POOL)]
    assert list(r["r_windows"]) == [8, 1]
    assert list(r["r_final"]) == [3, 0]
    assert r["idle_final"] == 0 and list(r["held_final"]) == [0, 0]


def pin_vetoed_donor_is_skipped(o):
    # M = 3, one GPU each, budget 3, R = (1, 1, 1), model 0 critical, models 1, 2
    # surplus (2.0, 3.0), instantaneous actuation, K = 1. The guard refuses
    # model 2 at tick 0.
    #  w0: donors 1 (Z 2) and 2 (Z 3, vetoed) -> donor 1
    #  w1: donor 1 is at its floor (R 0); donor 2 (no veto) -> donor 2
    # routable: (1,1,1) (2,0,1); final (3,0,0)
    S, f = _const_S(2, [0.2, 2.0, 3.0])
    r = o.control_act(_cfg(3, 2, 3), _prof([1, 1, 1]), S, f, _sc(1), 0, 0, veto=np.array([1 << 2, 0], np.uint64))
    assert _moves(r) == [(0, RES, 0, 1), (1, RES, 0, 2)]
    assert list(r["r_windows"]) == [3, 1, 2]
    assert list(r["r_final"]) == [3, 0, 0]
    free = o.control_act(_cfg(3, 2, 3), _prof([1, 1, 1]), S, f, _sc(1), 0, 0)
    assert _moves(free)[0] == (0, RES, 0, 2)  # without the veto the argmax donor is taken


def _random_scenarios(n, seed):
    rng = np.random.default_rng(seed)
    sc = np.zeros(n, O.SCENARIO_DTYPE)
    sc["max_moves"] = rng.choice([1, 2, 4, 8], n)
    sc["theta_scale"] = rng.uniform(0.5, 2.0, n)
    sc["tau_crit_override"] = np.where(rng.random(n) < 0.5, -1.0, rng.uniform(0.2, 0.8, n))
    return sc


def _trace_sets(o):
    """(cfg, prof, S, flags) of a few generated and hand-shaped traces."""
    out = []
    w = tg.standard(1).scaled(duration_ms=900_000)
    ev = w.generate(0, 1).trace(0)
    prof = O.pack_profiles(w.profile_columns(1))
    r = o.tss_trace(ev, w.window_ms, w.duration_ms, prof)
    out.append((w.trace_cfg(), prof, r["S"], r["flags"]))
    rng = np.random.default_rng(5)
    for i, M in enumerate((3, 6)):
        cfg = {"window_ms": 100, "duration_ms": 100 * 1500, "fast_period_ms": 300, "slow_period_ms": 700,
               "n_models": M, "budget": 3 * M + 4}
        ev = E.trace_random(50 + i, M, cfg["duration_ms"], 2500)
        p = np.zeros(M, O.PROFILE_DTYPE)
        p["w_p"], p["w_q"], p["alpha"] = rng.uniform(0.1, 0.9, M), rng.uniform(1, 3, M), rng.uniform(0.05, 1, M)
        p["theta"] = rng.uniform(20, 400, M)
        p["tau_crit"], p["tau_surplus"] = rng.uniform(0.2, 0.6, M), rng.uniform(1.1, 2.0, M)
        p["r_min"], p["r_init"] = rng.integers(0, 2, M), 2
        r = o.tss_trace(ev, cfg["window_ms"], cfg["duration_ms"], p)
        out.append((cfg, p, r["S"], r["flags"]))
    return out


def pin_instantaneous_actuation_reduces_to_the_base_rules(o):
    for t, (cfg, prof, S, flags) in enumerate(_trace_sets(o)):
        for i, sc in enumerate(_random_scenarios(60, 7 + t)):
            a = o.control(cfg, prof, S, flags, sc)
            b = o.control_act(cfg, prof, S, flags, sc, 0, 0)
            assert a["n_moves"] == b["n_moves"], (t, i)
            assert _moves(a) == _moves(b), (t, i)
            assert np.array_equal(a["r_final"], b["r_final"]) and np.array_equal(a["r_windows"], b["r_windows"])
            # unit footprints given explicitly and an all-clear veto table change nothing
            n_ticks = sum(1 for w in range(cfg["duration_ms"] // cfg["window_ms"])
                          if ((w + 1) * cfg["window_ms"]) % cfg["fast_period_ms"] == 0
                          or ((w + 1) * cfg["window_ms"]) % cfg["slow_period_ms"] == 0)
            c = o.control_act(cfg, prof, S, flags, sc, 0, 0, footprint=np.ones(len(prof), np.int32),
                              veto=np.zeros(n_ticks, np.uint64))
            assert _moves(c) == _moves(b) and np.array_equal(c["r_windows"], b["r_windows"])


def pin_gpu_conservation_and_move_bound_with_delays_footprints_vetoes(o):
    rng = np.random.default_rng(9)
    for t, (cfg, prof, S, flags) in enumerate(_trace_sets(o)):
        M = len(prof)
        nW = cfg["duration_ms"] // cfg["window_ms"]
        ticks = [w for w in range(nW) if ((w + 1) * cfg["window_ms"]) % cfg["fast_period_ms"] == 0
                 or ((w + 1) * cfg["window_ms"]) % cfg["slow_period_ms"] == 0]
        for i, sc in enumerate(_random_scenarios(20, 20 + t)):
            g = rng.integers(1, 4, M).astype(np.int32)
            cfg2 = dict(cfg)
            cfg2["budget"] = int((g * prof["r_init"]).sum() + rng.integers(0, 6))
            veto = rng.integers(0, 1 << M, len(ticks)).astype(np.uint64) & np.uint64(rng.integers(0, 2) * ((1 << M) - 1))
            r = o.control_act(cfg2, prof, S, flags, sc, int(rng.integers(0, 30)), int(rng.integers(0, 30)),
                              footprint=g, veto=veto)
            assert r["idle_final"] >= 0
            assert r["idle_final"] + int((g * r["r_final"]).sum()) + int(r["held_final"].sum()) == cfg2["budget"]
            assert (r["r_final"] >= 0).all()
            per_tick = {}
            for m in r["moves"]:
                per_tick[int(m["window"])] = per_tick.get(int(m["window"]), 0) + 1
                assert int(m["window"]) in ticks
                assert int(m["donor"]) == O.POOL or not ((int(veto[ticks.index(int(m["window"]))]) >> int(m["donor"])) & 1)
            assert all(v <= int(sc["max_moves"]) for v in per_tick.values())


def pin_bad_arguments_are_rejected(o):
    S, f = _const_S(3, [0.2, 2.0])
    for kw in ({"wake_w": -1, "sleep_w": 0}, {"wake_w": 0, "sleep_w": 0, "footprint": np.array([0, 1])},
               {"wake_w": 0, "sleep_w": 0, "footprint": np.array([2, 2])}):  # the last: above the GPU budget
        try:
            o.control_act(_cfg(2, 3, 3), _prof([1, 1]), S, f, _sc(1), **kw)
        except ValueError:
            continue
        raise AssertionError(f"accepted {kw}")


ALL = [pin_wake_delay_blocks_the_receiver_until_routable, pin_footprint_feasibility_picks_the_donor_and_blocks_later_moves,
       pin_larger_donor_returns_its_excess_after_the_sleep, pin_vetoed_donor_is_skipped,
       pin_instantaneous_actuation_reduces_to_the_base_rules,
       pin_gpu_conservation_and_move_bound_with_delays_footprints_vetoes, pin_bad_arguments_are_rejected]
