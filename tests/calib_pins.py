"""Pins of the calibration-sweep oracle (oracle/tre_oracle_calib.c).

Each pin takes an ``oracle.Oracle`` and raises AssertionError when the
oracle disagrees with a value fixed independently of it: hand-derived
latencies, counts and boundaries for small hand-built traces (derivations
in the comments), a brute-force statement of the boundary fit on small
random sets, a second implementation of the per-request join with numpy
scatter operations on generated traces, special cases that reduce to
closed forms, monotonicity, and conservation of judged requests.

Readings followed (paper, Section "Smoothing, Normalization, and
Calibration" and the SLO background): TTFT / TPOT / E2E from the first
DECODE and FINISH events of a request, attainment by arrival window, a
window healthy when ok >= q * judged, theta the smallest smoothed TSS whose
candidates at or above it are healthy at a rate of at least rho.
"""
import math

import numpy as np

import oracle as O
import tracegen as tg

A, P, D, F, ADMIT = 0, 1, 2, 3, 0x80


def _trace(rows):
    rows = sorted(rows, key=lambda r: r[0])  # stable: lifecycle order kept on equal ts
    cols = {"ts": np.array([r[0] for r in rows], np.int64), "model": np.array([r[1] for r in rows], np.uint8),
            "req": np.array([r[2] for r in rows], np.uint32), "type": np.array([r[3] for r in rows], np.uint8),
            "tokens": np.array([r[4] for r in rows], np.uint16)}
    return cols


def _slo(rows):
    a = np.zeros(len(rows), O.SLO_DTYPE)
    for i, r in enumerate(rows):
        a[i] = r
    return a


HAND = [
    # req 0, model 0: TTFT 60-10 = 50, E2E 150-10 = 140; DECODE tokens 24+24+10,
    # 34 after the first chunk: TPOT (150-60)/34
    (10, 0, 0, A, 100), (10, 0, 0, P | ADMIT, 100), (60, 0, 0, D, 24), (110, 0, 0, D, 24),
    (150, 0, 0, D, 10), (150, 0, 0, F, 0),
    # req 1, model 1: TTFT 250-20 = 230 = E2E; one DECODE event, no TPOT sample
    (20, 1, 1, A, 50), (30, 1, 1, P | ADMIT, 50), (250, 1, 1, D, 5), (250, 1, 1, F, 0),
    # req 2, model 0, arrives in window 1: TTFT 300-120 = 180, E2E 210, TPOT 30/24
    (120, 0, 2, A, 10), (130, 0, 2, P | ADMIT, 10), (300, 0, 2, D, 24), (330, 0, 2, D, 24), (330, 0, 2, F, 0),
    # req 3, model 0: no FINISH before the end -> censored
    (150, 0, 3, A, 10), (150, 0, 3, P | ADMIT, 10), (990, 0, 3, D, 24),
    # req 4, model 1: only an ARRIVE -> censored
    (900, 1, 4, A, 10),
    # req 6, model 1 (id 5 unused), window 1: TTFT 25, E2E 35, TPOT 10/24
    (105, 1, 6, A, 8), (105, 1, 6, P | ADMIT, 8), (130, 1, 6, D, 24), (140, 1, 6, D, 24), (140, 1, 6, F, 0),
    # req 9 is beyond req_cap = 8: ignored and counted
    (500, 1, 9, A, 8),
]
# model 0: TTFT <= 100, TPOT <= 2, E2E <= 200; model 1: TTFT <= 230 (met with
# equality by req 1), TPOT <= 0.1, E2E <= 300
HAND_SLO = [(100.0, 2.0, 200.0, 0.95, 0.9), (230.0, 0.1, 300.0, 0.95, 0.9)]


def pin_hand_trace_latencies_and_attainment(o):
    r = o.calib_requests(_trace(HAND), 100, 1000, _slo(HAND_SLO), 8)
    q = r["reqs"]
    assert r["bad_ids"] == 1
    assert [int(x) for x in q["complete"]] == [1, 1, 1, 0, 0, 0, 1, 0]
    assert [int(x) for x in q["model"]] == [0, 1, 0, 0, 1, -1, 1, -1]
    assert (int(q[0]["ttft_ms"]), int(q[0]["e2e_ms"])) == (50, 140) and q[0]["tpot_ms"] == 90.0 / 34.0
    assert (int(q[1]["ttft_ms"]), int(q[1]["e2e_ms"]), int(q[1]["has_tpot"])) == (230, 230, 0)
    assert (int(q[2]["ttft_ms"]), int(q[2]["e2e_ms"])) == (180, 210) and q[2]["tpot_ms"] == 30.0 / 24.0
    assert (int(q[6]["ttft_ms"]), int(q[6]["e2e_ms"])) == (25, 35) and q[6]["tpot_ms"] == 10.0 / 24.0
    # req 0 misses TPOT (2.65 > 2), req 2 misses TTFT, req 1 meets all (TTFT
    # bound met with equality), req 6 misses TPOT
    assert [int(x) for x in q["ok"]] == [0, 1, 0, 0, 0, 0, 0, 0]
    exp_j = np.zeros((2, 10), np.uint32)
    exp_ok = np.zeros((2, 10), np.uint32)
    exp_j[0, 0] = exp_j[0, 1] = 1      # req 0 (t 10), req 2 (t 120)
    exp_j[1, 0] = exp_j[1, 1] = 1      # req 1 (t 20), req 6 (t 105)
    exp_ok[1, 0] = 1
    assert np.array_equal(r["judged"], exp_j) and np.array_equal(r["ok"], exp_ok)


def _fit_one(o, S, healthy, judged=None, flags=None, q=0.95, rho=0.9):
    """Fit for one model from per-window S and health (ok = judged or 0)."""
    S = np.asarray(S, np.float64)
    n = S.shape[0]
    judged = np.ones(n, np.uint32) if judged is None else np.asarray(judged, np.uint32)
    ok = np.where(np.asarray(healthy, bool), judged, 0).astype(np.uint32)
    flags = np.full(n, O.INIT, np.uint8) if flags is None else np.asarray(flags, np.uint8)
    slo = _slo([(1.0, 1.0, 1.0, q, rho)])
    return o.calib_fit(S.reshape(n, 1), flags.reshape(n, 1), judged.reshape(1, n), ok.reshape(1, n), slo)[0]


def pin_hand_fit_with_ties(o):
    # S = 5 4 3 3 1 (by value) with health h h h u u. Walking down: 5 -> 1/1,
    # 4 -> 2/2, the pair at 3 together -> 3/4 = 0.75, 1 -> 3/5.
    S, h = [5.0, 3.0, 3.0, 1.0, 4.0], [1, 1, 0, 0, 1]
    f = _fit_one(o, S, h, rho=0.75)
    assert (f["theta"], int(f["n_above"]), int(f["healthy_above"])) == (3.0, 4, 3)
    assert (int(f["n_cand"]), int(f["n_healthy"])) == (5, 3)
    f = _fit_one(o, S, h, rho=0.8)  # 0.75 no longer reaches it: back to 4
    assert (f["theta"], int(f["n_above"]), int(f["healthy_above"])) == (4.0, 2, 2)
    # the healthy member of the tie alone (3/3) would pass 0.8, but a
    # threshold covers the whole tie
    f = _fit_one(o, [2.0, 2.0, 9.0], [0, 1, 1], rho=0.7)
    assert f["theta"] == 9.0 and int(f["n_above"]) == 1
    # non-candidates: no judged request, not initialised, idle
    f = _fit_one(o, [1.0, 2.0, 3.0, 4.0], [0, 0, 0, 1], judged=[1, 0, 1, 1],
                 flags=[O.INIT, O.INIT, 0, O.INIT | O.IDLE], rho=0.5)
    assert int(f["n_cand"]) == 1 and math.isinf(f["theta"]) and int(f["n_above"]) == 0


def pin_hand_ordering_counts(o):
    # The ordering check (RQ1): pairs of candidate windows with different S,
    # one healthy (h) and one not (u). S = 5h 4h 3h 3u 1u:
    #   concordant (larger S healthy): 5h>3u 5h>1u 4h>3u 4h>1u 3h>1u = 5
    #   discordant (larger S unhealthy): none (the unhealthy 3 ties with the
    #   healthy 3, and no healthy window lies below 3)
    f = _fit_one(o, [5.0, 3.0, 3.0, 1.0, 4.0], [1, 1, 0, 0, 1], rho=0.75)
    assert (int(f["concordant"]), int(f["discordant"])) == (5, 0)
    # S = 9u 7h 7u 2h: concordant none (no unhealthy window lies below a
    # healthy one); discordant 9u>7h, 9u>2h, 7u>2h = 3; the tie 7h/7u is in
    # neither (h * u = 2 * 2 = 4 = 0 + 3 + 1)
    f = _fit_one(o, [7.0, 9.0, 2.0, 7.0], [1, 0, 1, 0], rho=0.5)
    assert (int(f["concordant"]), int(f["discordant"])) == (0, 3)
    # perfectly ordered: every healthy window above every unhealthy one
    f = _fit_one(o, [10.0, 8.0, 6.0, 1.0, 0.5], [1, 1, 1, 0, 0], rho=0.5)
    assert (int(f["concordant"]), int(f["discordant"])) == (6, 0)
    # all one value of S: no pair counts either way
    f = _fit_one(o, [2.0, 2.0, 2.0], [1, 0, 1], rho=0.5)
    assert (int(f["concordant"]), int(f["discordant"])) == (0, 0)
    # only healthy windows
    f = _fit_one(o, [1.0, 2.0, 3.0], [1, 1, 1], rho=0.5)
    assert (int(f["concordant"]), int(f["discordant"])) == (0, 0)


def pin_window_health_threshold(o):
    # 19 of 20 meet the bound: healthy at q = 0.95 (equality), not at 0.951
    S = np.array([[1.0]])
    fl = np.array([[O.INIT]], np.uint8)
    j = np.array([[20]], np.uint32)
    ok = np.array([[19]], np.uint32)
    f = o.calib_fit(S, fl, j, ok, _slo([(1, 1, 1, 0.95, 1.0)]))[0]
    assert int(f["n_healthy"]) == 1 and f["theta"] == 1.0
    f = o.calib_fit(S, fl, j, ok, _slo([(1, 1, 1, 0.951, 1.0)]))[0]
    assert int(f["n_healthy"]) == 0 and math.isinf(f["theta"])


def _brute_fit(S, flags, judged, ok, q, rho):
    cand = [(S[w], ok[w] >= q * judged[w]) for w in range(len(S))
            if judged[w] >= 1 and (flags[w] & O.INIT) and not (flags[w] & O.IDLE)]
    best = (math.inf, 0, 0)
    for s, _ in cand:
        N = sum(1 for t, _ in cand if t >= s)
        H = sum(1 for t, h in cand if t >= s and h)
        if H >= rho * N and s < best[0]:
            best = (s, N, H)
    # every ordered pair of candidates with S_i > S_j, by the health of each
    conc = sum(1 for si, hi in cand for sj, hj in cand if si > sj and hi and not hj)
    disc = sum(1 for si, hi in cand for sj, hj in cand if si > sj and not hi and hj)
    return best, len(cand), sum(1 for _, h in cand if h), (conc, disc)


def pin_fit_matches_brute_force(o):
    rng = np.random.default_rng(31)
    for it in range(300):
        n = int(rng.integers(1, 40))
        M = int(rng.integers(1, 4))
        vals = rng.choice([0.5, 1.0, 1.5, 2.0, 3.25, 7.0, 1e-3, 1e4], 6) if it % 2 else rng.uniform(0, 10, 6)
        S = rng.choice(vals, (n, M))
        flags = rng.choice(np.array([O.INIT, O.INIT, O.INIT, 0, O.INIT | O.IDLE], np.uint8), (n, M))
        judged = rng.integers(0, 6, (M, n)).astype(np.uint32)
        ok = np.minimum(judged, rng.integers(0, 6, (M, n))).astype(np.uint32)
        slo = _slo([(1, 1, 1, float(rng.choice([0.0, 0.5, 0.8, 0.95, 1.0])), float(rng.choice([0.0, 0.3, 0.5, 0.9, 1.0, 1.1])))
                    for _ in range(M)])
        fit = o.calib_fit(S, flags, judged, ok, slo)
        for m in range(M):
            (th, N, H), nc, nh, (conc, disc) = _brute_fit(S[:, m], flags[:, m], judged[m].astype(float),
                                                          ok[m].astype(float), slo[m]["attain_q"],
                                                          slo[m]["reliability"])
            got = fit[m]
            assert (got["theta"], int(got["n_above"]), int(got["healthy_above"])) == (th, N, H), (it, m)
            assert (int(got["n_cand"]), int(got["n_healthy"])) == (nc, nh), (it, m)
            assert (int(got["concordant"]), int(got["discordant"])) == (conc, disc), (it, m)


def _numpy_join(ev, window_ms, nW, M, slo, req_cap):
    """The per-request join stated with numpy scatter operations."""
    n = ev["ts"].shape[0]
    rows = np.arange(n, dtype=np.int64)
    req = ev["req"].astype(np.int64)
    kind = ev["type"] & 3
    keep = req < req_cap
    big = np.int64(1) << 62

    def first(kd):
        out = np.full(req_cap, big, np.int64)
        sel = keep & (kind == kd)
        np.minimum.at(out, req[sel], rows[sel])
        return out

    a, f, e = first(A), first(D), first(F)
    dsum = np.zeros(req_cap, np.int64)
    sel = keep & (kind == D)
    np.add.at(dsum, req[sel], ev["tokens"][sel].astype(np.int64))
    done = (a < big) & (f < big) & (e < big)
    idx = np.nonzero(done)[0]
    ts = ev["ts"]
    ttft = ts[f[idx]] - ts[a[idx]]
    e2e = ts[e[idx]] - ts[a[idx]]
    rest = dsum[idx] - ev["tokens"][f[idx]].astype(np.int64)
    with np.errstate(divide="ignore", invalid="ignore"):
        tpot = np.where(rest > 0, (ts[e[idx]] - ts[f[idx]]).astype(np.float64) / np.maximum(rest, 1).astype(np.float64), 0.0)
    m = ev["model"][a[idx]].astype(np.int64)
    good = (ttft.astype(np.float64) <= slo["ttft_ms"][m]) & (e2e.astype(np.float64) <= slo["e2e_ms"][m]) & \
        ((rest == 0) | (tpot <= slo["tpot_ms"][m]))
    w = ts[a[idx]] // window_ms
    judged = np.zeros((M, nW), np.int64)
    okc = np.zeros((M, nW), np.int64)
    np.add.at(judged, (m, w), 1)
    np.add.at(okc, (m, w), good.astype(np.int64))
    return {"idx": idx, "ttft": ttft, "e2e": e2e, "tpot": tpot, "has_tpot": rest > 0, "good": good,
            "judged": judged, "ok": okc, "bad": int((~keep).sum())}


def _generated():
    out = []
    w = tg.standard(0)
    out.append((w, w.generate(0, 1).trace(0)))
    w = tg.standard(1).scaled(duration_ms=600_000)
    out.append((w, w.generate(0, 1).trace(0)))
    return out


def pin_join_matches_numpy_on_generated_traces(o):
    for w, ev in _generated():
        M, nW = w.n_models, w.n_windows
        slo = O.pack_slo(w.slo_columns(1))
        cap = int(ev["req"].max()) + 1
        for req_cap in (cap, cap // 2):  # the second drops the upper half of the ids
            r = o.calib_requests(ev, w.window_ms, w.duration_ms, slo, req_cap)
            x = _numpy_join(ev, w.window_ms, nW, M, slo, req_cap)
            q = r["reqs"]
            assert r["bad_ids"] == x["bad"]
            assert np.array_equal(np.nonzero(q["complete"])[0], x["idx"])
            qi = q[x["idx"]]
            assert np.array_equal(qi["ttft_ms"], x["ttft"]) and np.array_equal(qi["e2e_ms"], x["e2e"])
            assert np.array_equal(qi["has_tpot"].astype(bool), x["has_tpot"])
            assert np.array_equal(qi["tpot_ms"][x["has_tpot"]], x["tpot"][x["has_tpot"]])
            assert np.array_equal(qi["ok"].astype(bool), x["good"])
            assert np.array_equal(r["judged"], x["judged"]) and np.array_equal(r["ok"], x["ok"])
            # some requests pass and some fail on these traces
            assert 0 < int(r["ok"].sum()) < int(r["judged"].sum())


def pin_judged_requests_are_the_finished_ones(o):
    # generated requests always ARRIVE, DECODE at least once, then FINISH, so
    # the judged requests are exactly those whose FINISH is in the trace
    for w, ev in _generated():
        slo = O.pack_slo(w.slo_columns(1))
        r = o.calib_requests(ev, w.window_ms, w.duration_ms, slo, int(ev["req"].max()) + 1)
        n_fin = int(np.sum((ev["type"] & 3) == F))
        assert int(r["judged"].sum()) == n_fin == int(r["reqs"]["complete"].sum())
        assert (r["ok"] <= r["judged"]).all()
        # per model: judged requests are that model's FINISH events
        fin_m = np.bincount(ev["model"][(ev["type"] & 3) == F], minlength=w.n_models)
        assert np.array_equal(r["judged"].sum(axis=1), fin_m)


def pin_special_cases(o):
    for w, ev in _generated():
        M = w.n_models
        prof = O.pack_profiles(w.profile_columns(1))
        cap = int(ev["req"].max()) + 1
        slo = O.pack_slo(w.slo_columns(1))
        loose = slo.copy()
        loose["ttft_ms"] = loose["tpot_ms"] = loose["e2e_ms"] = np.inf
        r = o.calib_requests(ev, w.window_ms, w.duration_ms, loose, cap)
        assert np.array_equal(r["ok"], r["judged"])  # no bound: every judged request meets it
        tss = o.tss_trace(ev, w.window_ms, w.duration_ms, prof)
        S, fl = tss["S"], tss["flags"]
        cand = (r["judged"].T >= 1) & ((fl & O.INIT) != 0) & ((fl & O.IDLE) == 0)
        r = o.calib_requests(ev, w.window_ms, w.duration_ms, slo, cap)
        for q, rho in ((0.0, 0.9), (0.95, 0.0)):
            s2 = slo.copy()
            s2["attain_q"], s2["reliability"] = q, rho
            fit = o.calib_fit(S, fl, r["judged"], r["ok"], s2)
            for m in range(M):
                # every window healthy, or no reliability asked: the smallest candidate
                assert fit[m]["theta"] == S[cand[:, m], m].min() and int(fit[m]["n_above"]) == int(cand[:, m].sum())
        s2 = slo.copy()
        s2["reliability"] = 1.01
        fit = o.calib_fit(S, fl, r["judged"], r["ok"], s2)
        assert np.isinf(fit["theta"]).all() and (fit["n_above"] == 0).all()


def pin_monotone_in_reliability_and_bounds(o):
    for w, ev in _generated():
        prof = O.pack_profiles(w.profile_columns(1))
        cap = int(ev["req"].max()) + 1
        slo = O.pack_slo(w.slo_columns(1))
        tss = o.tss_trace(ev, w.window_ms, w.duration_ms, prof)
        prev_ok = None
        for scale in (0.5, 1.0, 2.0):
            s2 = slo.copy()
            for k in ("ttft_ms", "tpot_ms", "e2e_ms"):
                s2[k] = slo[k] * scale
            r = o.calib_requests(ev, w.window_ms, w.duration_ms, s2, cap)
            if prev_ok is not None:
                assert (r["ok"] >= prev_ok).all()  # looser bounds never fail more requests
            prev_ok = r["ok"]
        r = o.calib_requests(ev, w.window_ms, w.duration_ms, slo, cap)
        prev = None
        for rho in (0.0, 0.3, 0.6, 0.8, 0.9, 0.95, 1.0):
            s2 = slo.copy()
            s2["reliability"] = rho
            th = o.calib_fit(tss["S"], tss["flags"], r["judged"], r["ok"], s2)["theta"]
            if prev is not None:
                assert (th >= prev).all()  # asking for more reliability never lowers theta
            prev = th


def pin_bad_arguments_are_rejected(o):
    ev = _trace(HAND)
    for args in ((0, 1000), (100, 1050)):
        try:
            o.calib_requests(ev, args[0], args[1], _slo(HAND_SLO), 8)
        except ValueError:
            continue
        raise AssertionError(f"accepted window {args[0]} duration {args[1]}")


ALL = [pin_hand_trace_latencies_and_attainment, pin_hand_fit_with_ties, pin_hand_ordering_counts,
       pin_window_health_threshold,
       pin_fit_matches_brute_force, pin_join_matches_numpy_on_generated_traces,
       pin_judged_requests_are_the_finished_ones, pin_special_cases, pin_monotone_in_reliability_and_bounds,
       pin_bad_arguments_are_rejected]
