"""GPU parity of the calibration sweep (tre_calibrate) against the oracle.

For each trace the per-request records (judged or not, model, TTFT, E2E,
TPOT bit for bit, SLO met), the per-window (judged, ok) counts, the count of
out-of-range request ids and the per-model fit (theta bit for bit and the
four counts) must equal the oracle's. The oracle's fit runs on the GPU's
smoothed TSS and flags (those are compared with the oracle's own TSS by the
TSS parity tests), with its own per-window counts.

Inputs: the tiny, bursty, diverse and stress workloads (short and whole
traces, so every key-per-thread variant of the fit runs), hand-built traces
with censored requests, id gaps and ids past req_cap, constant-load traces
whose TSS repeats (long runs of equal keys), and argument errors.
"""
import sys

import numpy as np
import pytest

import oracle as O
import tracegen as tg
import calib_pins as CP

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


def _slo_rows(slo_cols, t, M):
    a = np.zeros(M, O.SLO_DTYPE)
    for k in O.SLO_DTYPE.names:
        a[k] = slo_cols[k][t * M:(t + 1) * M]
    return a


def _check(lib, name, cfg, traces, prof_cols, slo_cols, req_cap, check_traces=None, tiers=None):
    tre, device, torch = lib
    M = cfg["n_models"]
    cols, off = _columns(torch, traces)
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
    prof = tre.pack(prof_cols, tre.PROFILE_DTYPE)
    slo = tre.pack(slo_cols, tre.SLO_DTYPE)
    tss = tre.tss_outputs(ev, which=("tss64", "flags"))
    tre.tre_eval_tss(ev, prof, tss)
    out = tre.calib_outputs(ev, req_cap, with_reqs=True)
    # every output and the workspace start as garbage: the counters, lists
    # and records are the library's to clear (the stream zeroes its trace's
    # counters, the fallback tiers reset those of the traces they take)
    for k in ("counts", "fit", "n_bad", "ws", "reqs"):
        out[k].view(torch.uint8).fill_(0xA5)
    tre.tre_calibrate(ev, slo, tss["tss64"], tss["flags"], out)
    torch.cuda.synchronize()
    S = tss["tss64"].cpu().numpy()
    fl = tss["flags"].cpu().numpy()
    counts = out["counts"].cpu().numpy().view(np.uint32)
    fit0 = tre.unpack_fit(out["fit"]).reshape(len(traces), M).copy()
    assert (fit0["concordant"] == 0).all() and (fit0["discordant"] == 0).all()
    # the same fits with the ordering counts
    tre.tre_calib_order(ev, slo, tss["tss64"], tss["flags"], out)
    fit = tre.unpack_fit(out["fit"]).reshape(len(traces), M)
    for k in ("theta", "n_cand", "n_healthy", "n_above", "healthy_above"):
        assert np.array_equal(np.ascontiguousarray(fit0[k]).view(np.uint8), np.ascontiguousarray(fit[k]).view(np.uint8)), f"{name}: {k} of the two fits"
    reqs = tre.unpack_reqs(out["reqs"]).reshape(len(traces), req_cap)
    o = O.get()
    bad_total = 0
    for t in (range(len(traces)) if check_traces is None else check_traces):
        slo_t = _slo_rows(slo_cols, t, M)
        r = o.calib_requests(traces[t], cfg["window_ms"], cfg["duration_ms"], slo_t, req_cap)
        bad_total += r["bad_ids"]
        what = f"{name} trace {t}"
        g, q = reqs[t], r["reqs"]
        arrived = q["model"] >= 0
        assert np.array_equal((g["flags"] & tre.TRE_REQ_ARRIVED) != 0, arrived), what
        assert np.array_equal(g["model"][arrived], q["model"][arrived].astype(np.uint8)), what
        done = q["complete"] == 1
        assert np.array_equal((g["flags"] & tre.TRE_REQ_COMPLETE) != 0, done), f"{what}: judged requests"
        assert np.array_equal(g["ttft_ms"][done].astype(np.int64), q["ttft_ms"][done]), f"{what}: TTFT"
        assert np.array_equal(g["e2e_ms"][done].astype(np.int64), q["e2e_ms"][done]), f"{what}: E2E"
        has = q["has_tpot"] == 1
        assert np.array_equal((g["flags"] & tre.TRE_REQ_TPOT) != 0, has), f"{what}: TPOT defined"
        assert np.array_equal(g["tpot_ms"][has].view(np.uint64), q["tpot_ms"][has].view(np.uint64)), f"{what}: TPOT"
        assert np.array_equal((g["flags"] & tre.TRE_REQ_OK) != 0, q["ok"] == 1), f"{what}: SLO met"
        assert np.array_equal(counts[t] >> 16, r["judged"]), f"{what}: judged per window"
        assert np.array_equal(counts[t] & 0xFFFF, r["ok"]), f"{what}: ok per window"
        ref = o.calib_fit(S[t], fl[t], r["judged"], r["ok"], slo_t)
        for k in ("n_cand", "n_healthy", "n_above", "healthy_above", "concordant", "discordant"):
            assert np.array_equal(fit[t][k], ref[k]), f"{what}: fit {k} {fit[t][k]} vs {ref[k]}"
        assert np.array_equal(fit[t]["theta"].view(np.uint64), ref["theta"].view(np.uint64)), \
            f"{what}: theta {fit[t]['theta']} vs {ref['theta']}"
    if check_traces is None:
        assert int(out["n_bad"].cpu().numpy()[0]) == bad_total, f"{name}: ids past req_cap"
    n_fb = tre.calib_fallback_traces(ev, out)
    say(f"{name}: traces redone by the larger stream table and by the chunked path: {n_fb}")
    if tiers is not None:
        assert n_fb == tiers, f"{name}: traces redone {n_fb}, expected {tiers}"
    ev.close()
    return fit


def _req_cap(traces):
    return max(int(t["req"].max()) + 1 if len(t["req"]) else 1 for t in traces)


def test_tiny(lib):
    w = tg.standard(0)
    traces = [w.generate(0, 1).trace(0)]
    _check(lib, "tiny", w.trace_cfg(), traces, w.profile_columns(1), w.slo_columns(1), _req_cap(traces))


def test_bursty_with_several_reliability_targets(lib):
    w = tg.standard(1)
    traces = [w.generate(0, 1).trace(0)]
    slo = w.slo_columns(1)
    for rho, q in ((0.98, 0.95), (0.5, 0.9), (0.0, 1.0), (1.0, 0.0)):
        s = dict(slo)
        s["reliability"] = np.full_like(slo["reliability"], rho)
        s["attain_q"] = np.full_like(slo["attain_q"], q)
        say(f"bursty rho {rho} q {q}")
        _check(lib, f"bursty-{rho}-{q}", w.trace_cfg(), traces, w.profile_columns(1), s, _req_cap(traces))


def test_diverse_short(lib):
    w = tg.standard(3).scaled(n_traces=6, duration_ms=3_600_000)
    h = w.generate(0, 6)
    traces = [h.trace(i) for i in range(6)]
    _check(lib, "diverse-short", w.trace_cfg(), traces, w.profile_columns(6), w.slo_columns(6), _req_cap(traces))


def test_stress_whole_traces(lib):
    """14400 windows: the widest fit variant (16 keys per thread)."""
    w = tg.standard(4).scaled(n_traces=5, n_scenarios=5)
    h = w.generate(0, 5)
    traces = [h.trace(i) for i in range(5)]
    _check(lib, "stress-5tr", w.trace_cfg(), traces, w.profile_columns(5), w.slo_columns(5), _req_cap(traces))


def test_req_cap_below_and_above_the_ids(lib):
    w = tg.standard(1).scaled(duration_ms=600_000)
    traces = [w.generate(0, 1).trace(0)]
    cap = _req_cap(traces)
    for rc in (cap // 3, cap, 2 * cap + 5):
        say(f"req_cap {rc} (ids up to {cap - 1})")
        _check(lib, f"cap-{rc}", w.trace_cfg(), traces, w.profile_columns(1), w.slo_columns(1), rc)


def test_hand_trace_and_empty_traces(lib):
    cfg = {"window_ms": 100, "duration_ms": 1000, "fast_period_ms": 100, "slow_period_ms": 200,
           "n_models": 2, "budget": 4}
    hand = CP._trace(CP.HAND)
    empty = {k: v[:0] for k, v in hand.items()}
    traces = [empty, hand, empty, hand]
    prof = {"w_p": np.full(8, 0.2), "w_q": np.full(8, 2.0), "alpha": np.full(8, 0.5), "theta": np.full(8, 10.0),
            "tau_crit": np.full(8, 0.5), "tau_surplus": np.full(8, 1.5), "r_min": np.ones(8, np.int32),
            "r_init": np.full(8, 2, np.int32)}
    slo_rows = np.array(CP.HAND_SLO * 4, dtype=object)
    slo = {k: np.array([r[i] for r in slo_rows], np.float64)
           for i, k in enumerate(("ttft_ms", "tpot_ms", "e2e_ms", "attain_q", "reliability"))}
    _check(lib, "hand", cfg, traces, prof, slo, 8)


def test_constant_load_runs_of_equal_keys(lib):
    """Steady traces give long runs of equal smoothed TSS (ties across many
    windows) and windows where every digit of the keys agrees."""
    M = 3
    cfg = {"window_ms": 1000, "duration_ms": 1000 * 5000, "fast_period_ms": 5000, "slow_period_ms": 10000,
           "n_models": M, "budget": 9}
    rows = []
    rid = 0
    for m in range(M):
        for i in range(4999):
            t0 = i * 1000 + 100 * m
            rows += [(t0, m, rid, CP.A, 10), (t0, m, rid, CP.P | CP.ADMIT, 10), (t0 + 50 + 10 * m, m, rid, CP.D, 5),
                     (t0 + 900, m, rid, CP.D, 5), (t0 + 900, m, rid, CP.F, 0)]
            rid += 1
    steady = CP._trace(rows)
    prof = {"w_p": np.full(M, 0.2), "w_q": np.full(M, 2.0), "alpha": np.full(M, 1.0), "theta": np.full(M, 10.0),
            "tau_crit": np.full(M, 0.5), "tau_surplus": np.full(M, 1.5), "r_min": np.ones(M, np.int32),
            "r_init": np.full(M, 3, np.int32)}
    slo = {"ttft_ms": np.array([60.0, 60.0, 60.0]), "tpot_ms": np.array([200.0, 100.0, 1000.0]),
           "e2e_ms": np.full(M, 1000.0), "attain_q": np.full(M, 0.95), "reliability": np.array([0.9, 0.0, 1.0])}
    fit = _check(lib, "steady", cfg, [steady], prof, slo, rid)
    say("steady fit", fit)


def _small_cfg(M=2):
    return {"window_ms": 100, "duration_ms": 10_000, "fast_period_ms": 100, "slow_period_ms": 200,
            "n_models": M, "budget": 4 * M}


def _small_prof(M, n_traces):
    n = M * n_traces
    return {"w_p": np.full(n, 0.2), "w_q": np.full(n, 2.0), "alpha": np.full(n, 0.5), "theta": np.full(n, 10.0),
            "tau_crit": np.full(n, 0.5), "tau_surplus": np.full(n, 1.5), "r_min": np.ones(n, np.int32),
            "r_init": np.full(n, 2, np.int32)}


def _small_slo(M, n_traces):
    return {"ttft_ms": np.full(M * n_traces, 600.0), "tpot_ms": np.full(M * n_traces, 40.0),
            "e2e_ms": np.full(M * n_traces, 2500.0), "attain_q": np.full(M * n_traces, 0.9),
            "reliability": np.full(M * n_traces, 0.8)}


def _complete(rid, m, t0, span, tok=24):
    """ARRIVE, ADMIT, two DECODE chunks and the FINISH of one request."""
    return [(t0, m, rid, CP.A, 40), (t0, m, rid, CP.P | CP.ADMIT, 40), (t0 + span // 3, m, rid, CP.D, tok),
            (t0 + span, m, rid, CP.D, tok // 2), (t0 + span, m, rid, CP.F, 0)]


def _crowded(n, rid0=0):
    """n requests in flight together (all arrive in the first 50 ms, finish
    after 8 s): more live records than the stream's table keeps."""
    rows = []
    for j in range(n):
        rows += _complete(rid0 + j, j % 2, j % 50, 8000 + (j % 300), tok=24 + j % 7)
    return CP._trace(rows)


def _turnover(n, live):
    """One arrival and one finish per ms with `live` requests in flight: the
    stream rebuilds its table every tile."""
    rows = []
    for j in range(n):
        rows += _complete(j, j % 2, j, live, tok=10 + j % 5)
    return CP._trace(rows)


def _filler(n_rows, t0, rid0, gap=5):
    """Complete requests (5 rows each, `gap` ms apart from t0) padded with
    PREFILL rows of the first one to exactly n_rows rows."""
    rows, rid = [], rid0
    for j in range(n_rows // 5):
        rows += _complete(rid, j % 2, t0 + gap * j, 3, tok=8)
        rid += 1
    pad = n_rows % 5
    if pad:
        if rid == rid0:
            rows += [(t0, 0, rid, CP.A, 8)] + [(t0, 0, rid, CP.P, 8)] * (pad - 1)
            rid += 1
        else:
            rows[1:1] = [(t0, 0, rid0, CP.P, 8)] * pad
    return rows, rid


# tile rows of the two stream tiers (768 threads x 2 rows, 1024 x 4) and a
# row that is a tile boundary of both
TILE1, TILE2 = 1536, 4096
BOTH = 12288


def _boundary_instant(n_fin, before, order="fin_first", boundary=TILE1):
    """n_fin requests whose FINISH and a last DECODE fall on one instant X
    whose rows start `before` rows ahead of row `boundary` (a tile boundary
    of the first tier by default, of both tiers at BOTH); at X the FINISH rows come all first
    ("fin_first"), after the DECODE rows ("dec_first") or each with its own
    DECODE behind it ("interleaved"). Filler requests before and after."""
    pre = boundary - before - 3 * n_fin
    assert pre >= 0, pre
    rows, rid = _filler(pre, 0, 0, gap=max(1, min(5, 5000 // max(1, pre // 5))))
    X = 6000
    fin, dec = [], []
    for j in range(n_fin):
        m = j % 2
        rows += [(1000 + j, m, rid, CP.A, 30), (1000 + j, m, rid, CP.P | CP.ADMIT, 30), (2000 + j, m, rid, CP.D, 24)]
        fin.append((X, m, rid, CP.F, 0))
        dec.append((X, m, rid, CP.D, 3 + j % 9))
        rid += 1
    if order == "fin_first":
        rows += fin + dec
    elif order == "dec_first":
        rows += dec + fin
    else:
        rows += [r for pair in zip(fin, dec) for r in pair]
    more, _ = _filler(1500, 7000, rid)
    return CP._trace(rows + more)


def _long_instant(n_dec=3):
    """200 FINISH rows at the last instant X of a tile, followed by more than
    a whole tile of DECODE rows at X (1300 requests in flight, n_dec DECODE
    rows each at X: 3 outlast a tile of the first stream tier, 4 one of the
    second)."""
    rows, rid = [], 0
    X = 6000
    a = []
    for j in range(200):
        m = j % 2
        rows += [(1000 + j, m, rid, CP.A, 30), (1000 + j, m, rid, CP.P | CP.ADMIT, 30), (2000 + j, m, rid, CP.D, 24)]
        a.append((X, m, rid, CP.F, 0))
        rid += 1
    b, bf = [], []
    for j in range(1300):
        m = j % 2
        rows += [(100 + j % 500, m, rid, CP.A, 30), (100 + j % 500, m, rid, CP.P | CP.ADMIT, 30)]
        b += [(X, m, rid, CP.D, 5)] * n_dec
        bf.append((6100 + j % 100, m, rid, CP.F, 0))
        rid += 1
    return CP._trace(rows + a + b + bf)


def test_stream_rebuild_and_instants(lib):
    """The stream's own paths, against the oracle: a table rebuilt every tile
    (2300 requests in flight); tiles with more FINISH rows than the judge
    queue holds (2000 requests finishing within 300 ms); FINISH rows at a
    tile's last instant
    judged after the next tile, with the last DECODE of the same request in
    that instant listed after its FINISH (so beyond the boundary), with all
    256 FINISH rows the stream defers, and with the DECODE rows first; and
    traces that do not start on a 4-row boundary."""
    M = 2
    traces = [_turnover(7000, 2300), _crowded(2000), _boundary_instant(200, 120), _boundary_instant(300, 256),
              _boundary_instant(250, 251, "interleaved"), _boundary_instant(250, 250, "dec_first"),
              _turnover(3000, 700)]
    say("rows", [len(t["ts"]) for t in traces])
    _check(lib, "stream-paths", _small_cfg(M), traces, _small_prof(M, len(traces)), _small_slo(M, len(traces)),
           _req_cap(traces), tiers=(0, 0))


def test_stream_fallback(lib):
    """Traces the first stream tier hands to the second (twice the records,
    tiles of TILE2 rows) and those the second hands to the chunked path: more
    requests in flight than a table keeps, more FINISH rows at a tile's last
    instant than a tier defers, an instant longer than a tile; mixed with
    traces the first tier finishes, with ids past req_cap."""
    M = 2
    traces = [_crowded(3300),                                  # second tier
              _crowded(6000),                                  # chunked: too many in flight
              _turnover(3000, 500),                            # first tier
              _boundary_instant(400, 300),                     # second tier: 300 FINISH deferred
              _boundary_instant(400, 300, boundary=BOTH),      # chunked: 300 deferred in both
              _long_instant(3),                                # second tier
              _long_instant(4),                                # chunked: instant longer than 4096 rows
              _turnover(2000, 300)]                            # first tier
    say("rows", [len(t["ts"]) for t in traces])
    cap = _req_cap(traces) - 5
    _check(lib, "fallback", _small_cfg(M), traces, _small_prof(M, len(traces)), _small_slo(M, len(traces)), cap, tiers=(6, 3))


def test_model_counts(lib):
    for M in (1, 2, 17, 64):  # 2 and 64: the fit in model pairs
        w = tg.Workload(name=f"m{M}", n_traces=2, model_classes=[["7B", "13B", "34B", "70B"][m % 4] for m in range(M)],
                        interactive=[m % 2 == 0 for m in range(M)], r_init=[2] * M, budget=2 * M,
                        window_ms=500, duration_ms=900_000, process="mmpp2", rate=[0.5] * M,
                        proc_params={"mmpp_mult": 6.0, "mmpp_dwell_s": 60.0}, seed=40 + M)
        h = w.generate(0, 2)
        traces = [h.trace(i) for i in range(2)]
        say(f"M {M}: {sum(len(t['ts']) for t in traces)} events")
        _check(lib, f"M{M}", w.trace_cfg(), traces, w.profile_columns(2), w.slo_columns(2), _req_cap(traces))


def test_argument_errors(lib):
    tre, device, torch = lib
    w = tg.standard(0)
    traces = [w.generate(0, 1).trace(0)]
    cols, off = _columns(torch, traces)
    cfg = w.trace_cfg()
    prof = tre.pack(w.profile_columns(1), tre.PROFILE_DTYPE)
    slo = tre.pack(w.slo_columns(1), tre.SLO_DTYPE)
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
    tss = tre.tss_outputs(ev, which=("tss64", "flags"))
    tre.tre_eval_tss(ev, prof, tss)
    out = tre.calib_outputs(ev, 100)
    bad = dict(out)
    bad["req_cap"] = 0
    with pytest.raises(tre.TreError) as e:
        tre.tre_calibrate(ev, slo, tss["tss64"], tss["flags"], bad)
    assert e.value.code == tre.TRE_EINVAL
    small = dict(out)
    small["ws"] = out["ws"][:64]
    with pytest.raises(tre.TreError) as e:
        tre.tre_calibrate(ev, slo, tss["tss64"], tss["flags"], small)
    assert e.value.code == tre.TRE_ENOMEM
    ev_noreq = tre.tre_load_events(cols["ts"], cols["model"], None, cols["type"], cols["tokens"], off, cfg)
    with pytest.raises(tre.TreError) as e:
        tre.tre_calibrate(ev_noreq, slo, tss["tss64"], tss["flags"], out)
    assert e.value.code == tre.TRE_EINVAL
    ev_noreq.close()
    # more windows than the fit holds
    long_cfg = dict(cfg, window_ms=10, duration_ms=10 * 20000, fast_period_ms=10, slow_period_ms=20)
    t2 = {k: v[:0] for k, v in traces[0].items()}
    cols2, off2 = _columns(torch, [t2])
    ev2 = tre.tre_load_events(cols2["ts"], cols2["model"], cols2["req"], cols2["type"], cols2["tokens"], off2, long_cfg)
    tss2 = tre.tss_outputs(ev2, which=("tss64", "flags"))
    out2 = tre.calib_outputs(ev2, 4)
    with pytest.raises(tre.TreError) as e:
        tre.tre_calibrate(ev2, slo, tss2["tss64"], tss2["flags"], out2)
    assert e.value.code == tre.TRE_ERANGE
    ev2.close()
    ev.close()


def _fit_cases(nW, seed):
    """Per-model synthetic smoothed TSS and window health, chosen to take
    every path of the fit: a clean threshold, health hovering at the target
    rate, long runs of equal values, a dense cluster with outliers (whole
    buckets to resolve, or the full sort), and one constant value."""
    rng = np.random.default_rng(seed)
    base = rng.uniform(1.0, 100.0, nW)
    return [(base, base > 40, 0.98),
            (base, rng.random(nW) < 0.9, 0.9),
            (rng.choice([1.0, 2.0, 3.5, 8.0], nW), rng.random(nW) < 0.7, 0.75),
            (np.where(rng.random(nW) < 0.02, 1e6, 5.0 + rng.random(nW) * 1e-9), rng.random(nW) < 0.9, 0.9),
            (np.full(nW, 7.0), rng.random(nW) < 0.95, 0.9),
            # health ordered by S with noise near the boundary: the buckets
            # holding both kinds are few (their keys gathered for the
            # ordering counts)
            (base, base + rng.normal(0.0, 3.0, nW) > 40, 0.95)]


@pytest.mark.parametrize("nW,seed,density", [(1000, 1, 1.0), (1000, 2, 1.0), (14400, 1, 1.0), (14400, 2, 1.0),
                                              (1000, 3, 0.35), (3000, 5, 0.5), (6000, 6, 0.5), (14400, 3, 0.35),
                                              (14400, 4, 0.6)])
def test_fit_paths_with_given_tss(lib, nW, seed, density):
    """tre_calibrate takes the smoothed TSS as an input: feed chosen values,
    with one request per (window, model) whose TTFT meets or misses the
    bound, so every window's health is set by hand. With density below 1 a
    (window, model) has its request with that probability (the others judge
    nothing and are no candidates): the fit of a model pair then keeps both
    models' keys side by side, where dense windows make it load the second
    model again."""
    tre, device, torch = lib
    cases = _fit_cases(nW, seed)
    M = len(cases)
    win = 100
    rows = []
    rid = 0
    present = np.random.default_rng(seed + 100).random((nW, M)) < density
    for w in range(nW):
        for m, (_, healthy, _) in enumerate(cases):
            if not present[w, m]:
                continue
            t0 = w * win + 5 * m
            first = 10 if healthy[w] else 60  # TTFT bound 30 ms
            rows += [(t0, m, rid, CP.A, 8), (t0, m, rid, CP.P | CP.ADMIT, 8), (t0 + first, m, rid, CP.D, 8),
                     (t0 + 70, m, rid, CP.D, 8), (t0 + 70, m, rid, CP.F, 0)]
            rid += 1
    ev_h = CP._trace(rows)
    cfg = {"window_ms": win, "duration_ms": win * (nW + 1), "fast_period_ms": win, "slow_period_ms": win,
           "n_models": M, "budget": M}
    cols, off = _columns(torch, [ev_h])
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
    nWe = ev.n_windows
    S = np.ones((nWe, M))
    for m, (sv, _, _) in enumerate(cases):
        S[:nW, m] = sv
    fl = np.full((nWe, M), tre.TRE_FLAG_INIT, np.uint8)
    slo_cols = {"ttft_ms": np.full(M, 30.0), "tpot_ms": np.full(M, 1e9), "e2e_ms": np.full(M, 1e9),
                "attain_q": np.full(M, 0.95), "reliability": np.array([c[2] for c in cases])}
    slo = tre.pack(slo_cols, tre.SLO_DTYPE)
    tss64 = torch.from_numpy(S.reshape(1, nWe, M).copy()).cuda()
    flags = torch.from_numpy(fl.reshape(1, nWe, M).copy()).cuda()
    out = tre.calib_outputs(ev, rid)
    tre.tre_calibrate(ev, slo, tss64, flags, out)
    fit0 = tre.unpack_fit(out["fit"]).copy()
    # the same TSS 8 bytes off a 16-byte boundary: one model per workgroup
    # (pairs need 16-byte TSS loads); the same fits
    shifted = torch.zeros(tss64.numel() + 1, dtype=torch.float64, device="cuda")
    shifted[1:] = tss64.reshape(-1)
    tss64_u = shifted[1:].view(tss64.shape)
    assert tss64_u.data_ptr() % 16 == 8
    tre.tre_calibrate(ev, slo, tss64_u, flags, out)
    fit_u = tre.unpack_fit(out["fit"]).copy()
    for k in ("theta", "n_cand", "n_healthy", "n_above", "healthy_above"):
        assert np.array_equal(np.ascontiguousarray(fit0[k]).view(np.uint8), np.ascontiguousarray(fit_u[k]).view(np.uint8)), k
    tre.tre_calib_order(ev, slo, tss64, flags, out)
    torch.cuda.synchronize()
    fit = tre.unpack_fit(out["fit"])
    for k in ("theta", "n_cand", "n_healthy", "n_above", "healthy_above"):
        assert np.array_equal(np.ascontiguousarray(fit0[k]).view(np.uint8), np.ascontiguousarray(fit[k]).view(np.uint8)), k
    o = O.get()
    slo_h = _slo_rows(slo_cols, 0, M)
    r = o.calib_requests(ev_h, win, cfg["duration_ms"], slo_h, rid)
    assert (r["judged"][:, :nW] == present.T).all()
    ref = o.calib_fit(S, fl, r["judged"], r["ok"], slo_h)
    for m in range(M):
        for k in ("n_cand", "n_healthy", "n_above", "healthy_above", "concordant", "discordant"):
            assert fit[m][k] == ref[m][k], (m, k, fit[m], ref[m])
        assert fit[m]["theta"].view(np.uint64) == ref[m]["theta"].view(np.uint64), (m, fit[m], ref[m])
    say(f"nW {nW} seed {seed}: theta {fit['theta']}")
    ev.close()
