"""Pins of the CPU oracle to facts fixed outside the oracle itself.

Every check takes an ``oracle.Oracle`` instance and raises AssertionError
when the oracle disagrees with the fact.  ``test_oracle_pins.py`` runs them
on the real oracle; ``test_oracle_mutants.py`` runs them on deliberately
broken copies of the oracle (compiled from edited source on the CPU) and
requires every copy to fail at least one pin.

Sources of truth used here:
  * the paper's printed prefill-heavy / decode-heavy pair (golden file
    ``paper_pair.json``, cited there);
  * hand-derived exact rationals for tiny traces (``hand_traces.json``);
  * closed forms (constant request counts, alpha = 1, Z = 1/2 semantics,
    the denominator floor);
  * an independent second definition of the window integrals (per-request
    interval overlap computed from request ids) and of the token tallies
    (numpy bincount);
  * invariants of the control rules (replica conservation, bounded moves,
    donor / receiver eligibility, rebalancing deferred by a rescue);
  * exhaustive enumeration of feasible receiver/donor pairs on tiny states.
"""
from __future__ import annotations

import json
import math
import os
from fractions import Fraction

import numpy as np

import oracle as O
import tracegen as tg

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _frac(s):
    if s is None:
        return None
    if s == "inf":
        return math.inf
    return Fraction(s)


def close(x: float, ref, rel=2e-15) -> bool:
    if ref == math.inf:
        return x == math.inf
    ref = float(ref)
    return abs(x - ref) <= rel * max(abs(ref), 1e-300) or x == ref


def events_from_rows(rows):
    a = np.array(rows, dtype=np.int64).reshape(-1, 5)
    return {"ts": a[:, 0].astype(np.int64), "model": a[:, 1].astype(np.uint8),
            "req": a[:, 2].astype(np.uint32), "type": a[:, 3].astype(np.uint8),
            "tokens": a[:, 4].astype(np.uint16)}


def profile_array(spec, M):
    if "profile_per_model" in spec:
        rows = spec["profile_per_model"]
    else:
        rows = [spec["profile"]] * M
    a = np.zeros(M, O.PROFILE_DTYPE)
    for m, r in enumerate(rows):
        for k in O.PROFILE_DTYPE.names:
            a[m][k] = r[k]
    return a


def scenario_array(spec):
    s = np.zeros(1, O.SCENARIO_DTYPE)
    s[0]["trace"] = 0
    for k in ("max_moves", "theta_scale", "tau_crit_override"):
        s[0][k] = spec["scenario"][k]
    return s


def load_hand():
    d = json.load(open(os.path.join(GOLDEN, "hand_traces.json")))
    by = {t["name"]: t for t in d["traces"]}
    for t in d["traces"]:
        if "events_from" in t:
            t["events"] = by[t["events_from"]]["events"]
    return d["traces"]


# --------------------------------------------------------------- hand traces
def pin_hand_traces(o):
    for t in load_hand():
        cfg = t["cfg"]
        M = cfg["n_models"]
        ev = events_from_rows(t["events"])
        prof = profile_array(t, M)
        r = o.tss_trace(ev, cfg["window_ms"], cfg["duration_ms"], prof)
        if "expected_cells" in t:
            for w, m, P, D, A, W, raw, S, Z, idle in t["expected_cells"]["rows"]:
                assert r["P"][w, m] == P and r["D"][w, m] == D, (t["name"], w, m, "tokens")
                assert r["A_int"][w, m] == A and r["W_int"][w, m] == W, (t["name"], w, m, "integrals")
                assert bool(r["flags"][w, m] & O.IDLE) == bool(idle), (t["name"], w, m, "idle")
                assert close(r["S"][w, m], _frac(S)), (t["name"], w, m, "S", r["S"][w, m], S)
                if raw is not None:
                    got = o.raw_tss(prof[m]["w_p"], prof[m]["w_q"], P, D, A, W, cfg["window_ms"])
                    assert close(got, _frac(raw)), (t["name"], w, m, "raw", got, raw)
        ctl = o.control(cfg, prof, r["S"], r["flags"], scenario_array(t))
        exp = t["expected_control"]
        got_moves = [[int(x["window"]), int(x["path"]), int(x["receiver"]), int(x["donor"])] for x in ctl["moves"]]
        assert got_moves == exp["moves"], (t["name"], got_moves, exp["moves"])
        assert list(ctl["r_final"]) == exp["r_final"], (t["name"], ctl["r_final"])
        assert list(ctl["r_windows"]) == exp["r_windows"], (t["name"], ctl["r_windows"])


# ------------------------------------------------------- the paper's pair
def pin_paper_pair(o):
    d = json.load(open(os.path.join(GOLDEN, "paper_pair.json")))
    wms = d["window_ms"]
    sec = wms / 1000

    def tss(case, w_p):
        c = d[case]
        P = round(c["prefill_tps"] * sec)
        D = round(c["decode_tps"] * sec)
        A = round(c["queue"] * wms)
        return o.raw_tss(w_p, 2.0, P, D, A, 0, wms)

    wp = d["w_p_checked"]
    hp, hd = tss("prefill_heavy", wp), tss("decode_heavy", wp)
    assert close(hp, Fraction(d["expected_tss_at_w_p"]["prefill_heavy"]), 1e-14), hp
    assert close(hd, Fraction(d["expected_tss_at_w_p"]["decode_heavy"]), 1e-14), hd
    assert hp < hd  # the degraded prefill-heavy case scores lower
    flip = 20018 / 87170.14
    assert tss("prefill_heavy", flip - 1e-4) < tss("decode_heavy", flip - 1e-4)
    assert tss("prefill_heavy", flip + 1e-4) > tss("decode_heavy", flip + 1e-4)
    # with every token counted alike and no per-request normalisation the
    # ordering is the wrong way round (aggregate TPS)
    agg_p = d["prefill_heavy"]["prefill_tps"] + d["prefill_heavy"]["decode_tps"]
    agg_d = d["decode_heavy"]["prefill_tps"] + d["decode_heavy"]["decode_tps"]
    assert agg_p > agg_d
    # w_p = 1 and a unit queue reduce Eq. (1) to aggregate TPS (floor of 1)
    one_p = o.raw_tss(1.0, 2.0, 28521, 10025, wms, 0, wms)
    assert close(one_p, Fraction(28521 + 10025, 10)), one_p


# --------------------------------------------------------- closed forms
def _single(o, events, M=1, window_ms=1000, duration_ms=1000, **pk):
    prof = np.zeros(M, O.PROFILE_DTYPE)
    base = dict(w_p=0.5, w_q=2.0, alpha=0.5, theta=10.0, tau_crit=0.5, tau_surplus=1.5, r_min=1, r_init=1)
    base.update(pk)
    for k, v in base.items():
        prof[k] = v
    return o.tss_trace(events_from_rows(events), window_ms, duration_ms, prof), prof


def pin_floor(o):
    # waiting only, average queue 1/2 request: the denominator floors at one
    # request, so raw = the token rate (paper: the raw inverse reads 1.0
    # under the signal's floor)
    r, _ = _single(o, [[500, 0, 0, 0, 0]], duration_ms=1000)
    # no tokens at all but someone waiting: raw 0, not idle
    assert r["W_int"][0, 0] == 500 and r["A_int"][0, 0] == 0
    assert r["S"][0, 0] == 0.0 and not (r["flags"][0, 0] & O.IDLE)
    assert close(o.raw_tss(0.5, 2.0, 0, 7, 0, 500, 1000), Fraction(7000, 1000))
    # denominator exactly at the floor and just above it
    assert close(o.raw_tss(0.5, 2.0, 0, 10, 1000, 0, 1000), 10)
    assert close(o.raw_tss(0.5, 2.0, 0, 10, 1500, 0, 1000), Fraction(20, 3))
    assert close(o.raw_tss(0.5, 3.0, 4, 0, 0, 1000, 1000), Fraction(2000, 3000))


def pin_closed_forms(o):
    # k requests active for the whole window: A_int = k * window
    for k in (1, 3, 7):
        ev = []
        for i in range(k):
            ev += [[0, 0, i, 0, 10], [0, 0, i, 129, 10]]
        r, _ = _single(o, ev, window_ms=500, duration_ms=2000)
        assert list(r["A_int"][:, 0]) == [k * 500] * 4
        assert list(r["W_int"][:, 0]) == [0] * 4
    # alpha = 1: S equals the raw ratio in every non-idle window
    ev = [[0, 0, 0, 0, 10], [100, 0, 0, 129, 10], [1200, 0, 0, 2, 24], [2500, 0, 0, 2, 24], [2600, 0, 0, 3, 0]]
    r, prof = _single(o, ev, window_ms=1000, duration_ms=4000, alpha=1.0)
    for w in range(3):
        raw = o.raw_tss(0.5, 2.0, r["P"][w, 0], r["D"][w, 0], r["A_int"][w, 0], r["W_int"][w, 0], 1000)
        assert r["S"][w, 0] == raw
    assert r["flags"][3, 0] & O.IDLE and r["S"][3, 0] == r["S"][2, 0]
    # a constant raw ratio keeps the smoothed value constant (to rounding)
    ev = [[0, 0, 0, 0, 10], [0, 0, 0, 129, 10]]
    for w in range(6):
        if w:
            ev.append([w * 1000 + 400, 0, 0, 1, 10])
        ev.append([w * 1000 + 500, 0, 0, 2, 24])
    r, _ = _single(o, ev, window_ms=1000, duration_ms=6000, alpha=0.3)
    s0 = r["S"][0, 0]
    assert close(s0, Fraction(1000 * 24 + 500 * 10, 1000))  # 0.5*10 + 24 tokens over 1 s, A = 1
    for w in range(1, 6):
        assert abs(r["S"][w, 0] - 29.0) <= 4 * np.spacing(29.0)
    # smoothing weights: alpha on the new raw value
    assert close(o.smooth(0.25, 8.0, 4.0), Fraction(5))
    assert close(o.smooth(0.75, 8.0, 4.0), Fraction(7))


def _tick_ctl(o, S_vals, r_init, budget, K=1, tau_c=0.5, tau_s=1.5, r_min=1, fast=1000, slow=1000,
              theta=1.0, theta_scale=1.0, override=-1.0, idle=None, windows=1):
    """Control over `windows` windows whose smoothed TSS rows are S_vals
    (list of rows, or one row repeated)."""
    M = len(r_init)
    S = np.array(S_vals, dtype=np.float64).reshape(-1, M)
    if S.shape[0] == 1 and windows > 1:
        S = np.repeat(S, windows, axis=0)
    flags = np.full(S.shape, O.INIT, np.uint8)
    if idle is not None:
        flags[np.array(idle, bool).reshape(S.shape)] = O.IDLE | O.INIT
    prof = np.zeros(M, O.PROFILE_DTYPE)
    prof["theta"] = theta
    prof["tau_crit"] = tau_c
    prof["tau_surplus"] = tau_s
    prof["r_min"] = r_min
    prof["r_init"] = r_init
    prof["alpha"] = 1.0
    sc = np.zeros(1, O.SCENARIO_DTYPE)
    sc["max_moves"] = K
    sc["theta_scale"] = theta_scale
    sc["tau_crit_override"] = override
    cfg = {"window_ms": 1000, "duration_ms": 1000 * S.shape[0], "fast_period_ms": fast,
           "slow_period_ms": slow, "n_models": M, "budget": budget}
    return o.control(cfg, prof, S, flags, sc)


def _mv(ctl):
    return [(int(x["window"]), int(x["path"]), int(x["receiver"]), int(x["donor"])) for x in ctl["moves"]]


def pin_normalisation(o):
    # Eq. (2): Z = S / (theta * scale); Z = 1/2 means half the healthy
    # service.  With tau_crit = 1/2 the boundary itself is not critical.
    c = _tick_ctl(o, [5.0, 100.0], [2, 2], 4, theta=10.0, tau_c=0.5)
    assert _mv(c) == [(0, O.REBALANCE, 0, 1)]          # Z = 0.5: nominal, below 1
    c = _tick_ctl(o, [5.0, 100.0], [2, 2], 4, theta=10.0, tau_c=0.5000001)
    assert _mv(c) == [(0, O.RESCUE, 0, 1)]             # now critical
    # boundary scale: theta 10 * scale 2 -> Z = 0.25
    c = _tick_ctl(o, [5.0, 100.0], [2, 2], 4, theta=10.0, tau_c=0.3, theta_scale=2.0)
    assert _mv(c) == [(0, O.RESCUE, 0, 1)]
    c = _tick_ctl(o, [5.0, 100.0], [2, 2], 4, theta=10.0, tau_c=0.3, theta_scale=0.5)
    assert _mv(c) == []                                # Z = 1: no deficit
    # rescue-threshold override replaces the profile's tau_crit
    c = _tick_ctl(o, [5.0, 100.0], [2, 2], 4, theta=10.0, tau_c=0.1, override=0.6)
    assert _mv(c) == [(0, O.RESCUE, 0, 1)]
    # surplus strictly above tau_surplus; Z equal to tau_surplus is nominal
    c = _tick_ctl(o, [1.0, 15.0, 16.0], [2, 2, 2], 6, theta=10.0, tau_c=0.5, tau_s=1.5)
    assert _mv(c) == [(0, O.RESCUE, 0, 2)]
    c = _tick_ctl(o, [1.0, 15.0, 14.0], [2, 2, 2], 6, theta=10.0, tau_c=0.5, tau_s=1.5)
    assert _mv(c) == [(0, O.RESCUE, 0, 1)]             # both nominal: the larger Z
    c = _tick_ctl(o, [1.0, 15.0, 14.5], [2, 2, 2], 6, theta=10.0, tau_c=0.5, tau_s=[1.5, 1.5, 1.4])
    assert _mv(c) == [(0, O.RESCUE, 0, 2)]             # Z = tau_surplus is not surplus


def pin_cadence(o):
    # fast every 2 windows, slow every 3 (not nested)
    # model 0 critical throughout: rescues at t = 2000, 4000, 6000 only;
    # the slow-only tick at 3000 is deferred
    c = _tick_ctl(o, [0.1, 100.0], [2, 9], 11, fast=2000, slow=3000, windows=6, K=1, r_min=1)
    assert _mv(c) == [(1, O.RESCUE, 0, 1), (3, O.RESCUE, 0, 1), (5, O.RESCUE, 0, 1)], _mv(c)
    # model 0 at Z = 0.8 (nominal, below 1): rebalances at slow ticks only
    c = _tick_ctl(o, [0.8, 100.0], [2, 9], 11, fast=2000, slow=3000, windows=6, K=1)
    assert _mv(c) == [(2, O.REBALANCE, 0, 1), (5, O.REBALANCE, 0, 1)], _mv(c)
    # replicas in force per window: moves take effect from the next window
    assert list(c["r_windows"]) == [2 * 3 + 3 * 3 + 0, 9 * 3 + 8 * 3]
    assert list(c["r_final"]) == [4, 7]
    # a critical model defers rebalancing of a different below-boundary model
    c = _tick_ctl(o, [0.1, 0.8, 100.0], [1, 2, 9], 12, fast=2000, slow=1000, windows=1, K=4)
    assert _mv(c) == []  # t = 1000: slow only, critical present -> nothing


def pin_control_rules(o):
    # receiver is the argmin; only one move per model per tick
    c = _tick_ctl(o, [0.3, 0.1, 0.2, 100.0, 90.0], [2, 2, 2, 2, 2], 10, K=4)
    mv = _mv(c)
    assert mv[0] == (0, O.RESCUE, 1, 3) and mv[1] == (0, O.RESCUE, 2, 4), mv
    assert len(mv) == 2   # model 0 has no donor left (both surplus donors used)
    # donor must be strictly healthier than the receiver
    c = _tick_ctl(o, [0.8, 0.8], [2, 2], 4, K=1)
    assert _mv(c) == []
    # donor floor: R > r_min
    c = _tick_ctl(o, [0.1, 100.0], [2, 2], 4, K=1, r_min=2)
    assert _mv(c) == []
    c = _tick_ctl(o, [0.1, 100.0], [2, 3], 5, K=1, r_min=2)
    assert _mv(c) == [(0, O.RESCUE, 0, 1)]
    # idle budget before any donor, then donors
    c = _tick_ctl(o, [0.1, 0.2, 100.0], [1, 1, 3], 6, K=3)
    assert _mv(c) == [(0, O.RESCUE, 0, O.POOL), (0, O.RESCUE, 1, 2)], _mv(c)
    assert list(c["r_final"]) == [2, 2, 2]
    # surplus donors before nominal ones, even when the nominal model has the
    # larger Z (possible with per-model surplus thresholds)
    c = _tick_ctl(o, [0.1, 1.4, 1.3], [2, 2, 2], 6, K=1, tau_s=[1.5, 1.5, 1.2])
    assert _mv(c) == [(0, O.RESCUE, 0, 2)]
    c = _tick_ctl(o, [0.1, 1.4, 1.3], [2, 2, 2], 6, K=1, tau_s=[1.5, 1.5, 1.5])
    assert _mv(c) == [(0, O.RESCUE, 0, 1)]
    # idle / uninitialised models read Z = inf: preferred donors, never receivers
    c = _tick_ctl(o, [0.1, 1.0, 7.0], [2, 2, 2], 6, K=1, idle=[[False, True, False]])
    assert _mv(c) == [(0, O.RESCUE, 0, 1)]
    # rebalancing path: receivers need Z < 1; with nothing below 1, no move
    c = _tick_ctl(o, [1.0, 1.2, 100.0], [2, 2, 2], 6, K=2)
    assert _mv(c) == []
    c = _tick_ctl(o, [0.99, 1.2, 100.0], [2, 2, 2], 6, K=2)
    assert _mv(c) == [(0, O.REBALANCE, 0, 2)]
    # replica conservation
    assert int(c["r_final"].sum()) == 6


# ------------------------------------------------------- tallies & integrals
def interval_integrals(ev, window_ms, duration_ms, M):
    """Independent second definition of the window integrals: each request
    contributes its waiting interval [arrive, admit) and its active interval
    [admit, finish); a missing end is the end of the trace.  Integral over a
    window = total overlap of the intervals with that window."""
    nW = duration_ms // window_ms
    kind = ev["type"] & 3
    admit = (ev["type"] & 0x80) != 0
    key = ev["req"].astype(np.int64)
    A = np.zeros((nW, M), np.int64)
    W = np.zeros((nW, M), np.int64)
    arrive_t, admit_t, fin_t, mod = {}, {}, {}, {}
    for t, r, k, ad, m in zip(ev["ts"].tolist(), key.tolist(), kind.tolist(), admit.tolist(), ev["model"].tolist()):
        mod[r] = m
        if k == 0:
            arrive_t[r] = t
        elif k == 1 and ad:
            admit_t[r] = t
        elif k == 3:
            fin_t[r] = t
    edges = np.arange(nW + 1, dtype=np.int64) * window_ms

    def add(arr, m, x, y):
        if y <= x:
            return
        lo = np.maximum(edges[:-1], x)
        hi = np.minimum(edges[1:], y)
        arr[:, m] += np.maximum(hi - lo, 0)

    for r, m in mod.items():
        a = arrive_t.get(r)
        s = admit_t.get(r)
        f = fin_t.get(r)
        if a is not None:
            add(W, m, a, s if s is not None else duration_ms)
        if s is not None:
            add(A, m, s, f if f is not None else duration_ms)
    return A, W


def _small_workloads():
    w0 = tg.standard(0)
    yield w0, 0
    yield w0.scaled(duration_ms=120_000, window_ms=250, seed=11), 0
    w1 = tg.standard(1).scaled(duration_ms=90_000)
    yield w1, 0
    w3 = tg.standard(3).scaled(duration_ms=40_000, n_traces=2)
    yield w3, 1
    w4 = tg.standard(4).scaled(duration_ms=60_000, n_traces=2, proc_params={
        "flash_mult": 10.0, "flash_len_s": 10.0, "flash_first_s": 20.0, "flash_every_s": 30.0,
        "flash_models": 4})
    yield w4, 1


def pin_integrals_and_tallies(o):
    for w, t in _small_workloads():
        evs = w.generate(t, t + 1, threads=2)
        ev = evs.trace(0)
        M = w.n_models
        prof = O.pack_profiles(w.profile_columns(1))
        r = o.tss_trace(ev, w.window_ms, w.duration_ms, prof)
        A, W = interval_integrals(ev, w.window_ms, w.duration_ms, M)
        assert np.array_equal(r["A_int"], A), (w.name, "A_int")
        assert np.array_equal(r["W_int"], W), (w.name, "W_int")
        nW = w.n_windows
        win = ev["ts"] // w.window_ms
        kind = ev["type"] & 3
        cell = win * M + ev["model"].astype(np.int64)
        tok = ev["tokens"].astype(np.int64)
        P = np.bincount(cell[kind == 1], weights=tok[kind == 1], minlength=nW * M).astype(np.int64)
        D = np.bincount(cell[kind == 2], weights=tok[kind == 2], minlength=nW * M).astype(np.int64)
        assert np.array_equal(r["P"].reshape(-1), P), (w.name, "P")
        assert np.array_equal(r["D"].reshape(-1), D), (w.name, "D")


def pin_monotone(o):
    # more served tokens never lower TSS (correctly rounded operations are
    # monotone, so this holds exactly, not just approximately)
    rng = np.random.default_rng(7)
    for _ in range(300):
        wp, wq = rng.uniform(0, 1), rng.uniform(1, 4)
        P, D = int(rng.integers(0, 5000)), int(rng.integers(0, 5000))
        A, W = int(rng.integers(0, 50000)), int(rng.integers(0, 50000))
        base = o.raw_tss(wp, wq, P, D, A, W, 1000)
        assert o.raw_tss(wp, wq, P + 1, D, A, W, 1000) >= base
        assert o.raw_tss(wp, wq, P, D + 1, A, W, 1000) > base
        assert o.raw_tss(wp, wq, P, D, A + 1000, W, 1000) <= base or A + wq * W < 1000
        assert o.raw_tss(wp, wq, P, D, A, W + 1000, 1000) <= base
        s = o.smooth(0.3, base, 10.0)
        assert o.smooth(0.3, o.raw_tss(wp, wq, P, D + 1, A, W, 1000), 10.0) >= s


# ------------------------------------------------------------ invariants
def check_control_invariants(cfg, prof, S, flags, sc, ctl):
    """Check one scenario's moves against the rules, replaying them."""
    M = cfg["n_models"]
    nW = cfg["duration_ms"] // cfg["window_ms"]
    theta = prof["theta"] * sc["theta_scale"]
    tau_c = np.full(M, sc["tau_crit_override"]) if sc["tau_crit_override"] >= 0 else prof["tau_crit"]
    R = prof["r_init"].astype(np.int64).copy()
    pool = cfg["budget"] - int(R.sum())
    moves = ctl["moves"]
    assert ctl["n_moves"] == len(moves)
    i = 0
    rw = np.zeros(M, np.int64)
    for w in range(nW):
        rw += R
        tick = [mv for mv in moves[i:] if mv["window"] == w]
        t_end = (w + 1) * cfg["window_ms"]
        fast = t_end % cfg["fast_period_ms"] == 0
        slow = t_end % cfg["slow_period_ms"] == 0
        Z = np.where((flags[w] & O.IDLE) | ((flags[w] & O.INIT) == 0), np.inf, S[w] / theta)
        crit = Z < tau_c
        surplus = Z > prof["tau_surplus"]
        if not (fast or slow):
            assert not tick
            continue
        if crit.any() and not fast:
            assert not tick, "rebalancing must wait while a rescue is pending"
        assert len(tick) <= sc["max_moves"]
        seen = set()
        for mv in tick:
            r, d, path = int(mv["receiver"]), int(mv["donor"]), int(mv["path"])
            if crit.any():
                assert path == O.RESCUE and crit[r]
            else:
                assert path == O.REBALANCE and slow and Z[r] < 1.0
            assert r not in seen
            # receiver: the lowest Z among eligible models not yet moved
            elig = [m for m in range(M) if m not in seen and (crit[m] if crit.any() else Z[m] < 1.0)]
            assert Z[r] == min(Z[m] for m in elig) and r == min(m for m in elig if Z[m] == Z[r])
            seen.add(r)
            if d == O.POOL:
                assert pool > 0
                pool -= 1
            else:
                assert pool == 0 and d not in seen and d != r
                assert R[d] > prof["r_min"][d] and Z[d] > Z[r] and not crit[d]
                cand = [m for m in range(M) if m not in seen and R[m] > prof["r_min"][m] and Z[m] > Z[r]]
                sur = [m for m in cand if surplus[m]]
                nom = [m for m in cand if not crit[m] and not surplus[m]]
                pick = sur if sur else nom
                best = max(Z[m] for m in pick)
                assert d == min(m for m in pick if Z[m] == best)
                R[d] -= 1
                seen.add(d)
            R[r] += 1
        i += len(tick)
        assert int(R.sum()) + pool == cfg["budget"]
    assert i == len(moves)
    assert np.array_equal(R, ctl["r_final"]) and np.array_equal(rw, ctl["r_windows"])


def pin_invariants(o):
    rng = np.random.default_rng(5)
    for w, t in _small_workloads():
        ev = w.generate(t, t + 1, threads=2).trace(0)
        prof = O.pack_profiles(w.profile_columns(1))
        r = o.tss_trace(ev, w.window_ms, w.duration_ms, prof)
        cfg = w.trace_cfg()
        for k in range(6):
            sc = np.zeros(1, O.SCENARIO_DTYPE)
            sc["max_moves"] = [1, 2, 4, 3, 1, 8][k]
            sc["theta_scale"] = rng.uniform(0.5, 2.0)
            sc["tau_crit_override"] = rng.uniform(0.2, 0.8) if k % 2 else -1.0
            p = prof.copy()
            if k >= 4:  # leave idle budget and vary floors
                cfg = dict(cfg, budget=cfg["budget"] + 3)
                p["r_min"] = rng.integers(0, 3, size=p.shape[0])
            ctl = o.control(cfg, p, r["S"], r["flags"], sc)
            check_control_invariants(cfg, p, r["S"], r["flags"], sc[0], ctl)


def pin_bruteforce(o):
    # single tick, K = 1: the chosen pair is the lexicographic optimum over
    # all feasible (receiver, source) pairs of
    #   (Z_receiver, receiver, source class [idle budget < surplus < nominal],
    #    -Z_source, source)
    rng = np.random.default_rng(11)
    for _ in range(400):
        M = int(rng.integers(1, 5))
        Zs = rng.choice([0.05, 0.3, 0.5, 0.7, 1.0, 1.2, 1.5, 2.0, np.inf], size=M)
        S = np.where(np.isinf(Zs), 1.0, Zs)
        idle = np.isinf(Zs)
        r_init = rng.integers(0, 4, size=M)
        extra = int(rng.integers(0, 2))
        slow = bool(rng.integers(0, 2))
        c = _tick_ctl(o, [S], r_init.tolist(), int(r_init.sum()) + extra, K=1, idle=[idle],
                      fast=1000, slow=1000 if slow else 2000)
        tau_c, tau_s = 0.5, 1.5
        crit = Zs < tau_c
        sur = Zs > tau_s
        best = None
        for r in range(M):
            if crit.any():
                ok = crit[r]
            else:
                ok = slow and Zs[r] < 1.0
            if not ok:
                continue
            srcs = []
            if extra > 0:
                srcs.append((0, 0.0, -1))
            else:
                for d in range(M):
                    if d == r or r_init[d] <= 1 or not Zs[d] > Zs[r] or crit[d]:
                        continue
                    srcs.append((1 if sur[d] else 2, -Zs[d], d))
            for s in srcs:
                key = (Zs[r], r) + s
                if best is None or key < best:
                    best = key
        mv = _mv(c)
        if best is None:
            assert mv == [], (Zs, r_init, extra, mv)
        else:
            d = O.POOL if best[4] == -1 else best[4]
            path = O.RESCUE if crit.any() else O.REBALANCE
            assert mv == [(0, path, best[1], d)], (Zs, r_init, extra, mv, best)


# ------------------------------------------------- counts never negative
def pin_state(o):
    """A_m(t) and W_m(t) of Eq. (1) are numbers of active and of waiting
    requests (Section "Design Rationale and Definition"), so a stream that
    takes either below zero at some instant is rejected. They are step
    functions: the rows that share one instant may come in any order, only
    the counts after the last of them are values of the functions. A
    request is admitted once (the ADMIT bit moves it from waiting to
    active), which the request ids make checkable."""
    ARR, PF, ADM, DEC, FIN = 0, 1, 0x81, 2, 3

    def st(rows, M=2):
        return o.trace_status(events_from_rows(rows), 100, 1000, M)

    life = [[10, 0, 1, ARR, 5], [20, 0, 1, ADM, 5], [30, 0, 1, DEC, 3], [40, 0, 1, FIN, 0]]
    assert st(life) == 0
    # FINISH with nothing active: A_0 = -1 on [15, 20)
    assert st([[10, 0, 1, ARR, 5], [15, 0, 1, FIN, 0], [20, 0, 1, ADM, 5]]) == -5
    # ADMIT with nothing waiting: W_0 = -1 while A_0 = 1
    assert st([[20, 0, 1, ADM, 5], [30, 0, 1, FIN, 0]]) == -5
    # the counts are per model: model 1 admits while only model 0 waits
    assert st([[10, 0, 1, ARR, 5], [20, 1, 2, ADM, 5]]) == -5
    # model 0 negative at an instant whose last row is model 1's
    assert st([[10, 0, 1, ADM, 5], [10, 1, 2, ARR, 5], [50, 1, 2, ADM, 5]]) == -5
    # negative at the last instant of the trace
    assert st([[10, 0, 1, ARR, 5], [20, 0, 1, ADM, 5], [999, 0, 1, FIN, 0], [999, 0, 1, FIN, 0]]) == -5
    # order is checked first: an unsorted stream is an order error
    assert st([[20, 0, 1, ADM, 5], [10, 0, 1, ARR, 5]]) == -2
    # rows of one instant out of lifecycle order (ADMIT listed before its
    # ARRIVE, FINISH before the ADMIT of the same instant): accepted, with
    # the tallies of the lifecycle order
    odd = [[10, 0, 1, ADM, 5], [10, 0, 1, ARR, 5], [50, 1, 2, ARR, 4], [60, 1, 2, FIN, 0], [60, 1, 2, ADM, 4],
           [70, 0, 1, FIN, 0]]
    canon = [[10, 0, 1, ARR, 5], [10, 0, 1, ADM, 5], [50, 1, 2, ARR, 4], [60, 1, 2, ADM, 4], [60, 1, 2, FIN, 0],
             [70, 0, 1, FIN, 0]]
    assert st(odd) == 0
    a, _ = _single(o, odd, M=2, window_ms=100, duration_ms=1000)
    b, _ = _single(o, canon, M=2, window_ms=100, duration_ms=1000)
    for k in ("P", "D", "A_int", "W_int", "flags"):
        assert np.array_equal(a[k], b[k]), k
    assert a["A_int"][0, 0] == 60 and a["W_int"][0, 1] == 10
    # request ids: an id admitted twice; a later non-admitting PREFILL is fine
    ev = events_from_rows([[10, 0, 7, ARR, 5], [11, 0, 8, ARR, 5], [20, 0, 7, ADM, 5], [21, 0, 7, ADM, 5],
                           [30, 0, 8, PF, 5]])
    assert o.check_admits(ev) == (-6, 7)
    ev = events_from_rows([[10, 0, 7, ARR, 5], [20, 0, 7, ADM, 5], [25, 0, 7, PF, 5], [30, 1, 9, ADM, 5],
                           [31, 1, 4, ADM, 5], [32, 1, 9, ADM, 5], [33, 0, 4, ADM, 5]])
    assert o.check_admits(ev) == (-6, 4)
    assert o.check_admits(events_from_rows(life)) == (0, None)
    assert o.check_admits(events_from_rows([[5, 0, 3, ADM, 1], [6, 0, 4, ADM, 1], [7, 0, 3, PF, 1]])) == (0, None)
    # request ids: a request arrives once, finishes once, and neither arrives
    # nor decodes after its FINISH (rows of its FINISH instant in any order)
    lc = lambda rows: o.check_lifecycle(events_from_rows(rows))
    assert lc(life) == (0, None)
    assert lc([[10, 0, 7, ARR, 5], [20, 0, 7, ARR, 5], [30, 0, 8, ARR, 5]]) == (-7, 7)
    assert lc([[10, 0, 3, ARR, 5], [40, 0, 3, FIN, 0], [50, 0, 3, FIN, 0]]) == (-7, 3)
    assert lc([[10, 0, 4, ARR, 5], [40, 0, 4, FIN, 0], [41, 0, 4, DEC, 2]]) == (-7, 4)
    assert lc([[40, 0, 5, FIN, 0], [41, 0, 5, ARR, 2]]) == (-7, 5)
    # the smallest offending id, not the first in row order
    assert lc([[10, 0, 9, ARR, 5], [11, 0, 9, ARR, 5], [12, 0, 2, FIN, 0], [13, 0, 2, FIN, 0]]) == (-7, 2)
    # accepted: a DECODE listed after the FINISH of the same instant, a
    # PREFILL or ADMIT after the FINISH, a DECODE before the ARRIVE, ids with
    # no ARRIVE or no FINISH
    assert lc([[10, 0, 1, ARR, 5], [40, 0, 1, FIN, 0], [40, 0, 1, DEC, 3]]) == (0, None)
    assert lc([[10, 0, 1, ARR, 5], [40, 0, 1, FIN, 0], [45, 0, 1, PF, 3], [46, 0, 1, ADM, 3]]) == (0, None)
    assert lc([[5, 0, 1, DEC, 2], [10, 0, 1, ARR, 5], [40, 0, 1, FIN, 0]]) == (0, None)
    assert lc([[5, 0, 1, DEC, 2], [9, 0, 1, FIN, 0], [12, 0, 2, ARR, 5], [30, 0, 2, DEC, 3]]) == (0, None)


ALL_PINS = [pin_hand_traces, pin_paper_pair, pin_floor, pin_closed_forms, pin_normalisation,
            pin_cadence, pin_control_rules, pin_integrals_and_tallies, pin_monotone,
            pin_invariants, pin_bruteforce, pin_state]
