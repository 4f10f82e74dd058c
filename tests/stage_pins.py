"""Pins of the stage-aware service-share oracle (oracle/tre_oracle_stage.c).

Each pin takes an ``oracle.Oracle`` and raises AssertionError when the
oracle disagrees with something fixed independently of it:
- a hand-built two-model trace whose per-window stage shares are derived
  below as exact rationals (floors binding and not, idle holds, a waiting
  request never admitted, the waiting weight w_q mattering);
- a model with no prompt tokens and no waiting time: its decode share is the
  base oracle's TSS bit for bit (Eq. (1) reduces to its decode part), and
  its prefill share is idle throughout;
- the mediant relation: wherever neither stage floor binds, Eq. (1)'s raw
  ratio (the base oracle, itself pinned) lies between the two stage ratios
  and equals (num_p + num_d) / (den_p + den_d);
- special cases: alpha = 1 makes each share the raw ratio of its last busy
  window; k requests each served r decode tokens per second over the whole
  window give a decode share of r;
- monotonicity: more decode tokens never lower the decode share, more
  waiting never raises the prefill share.

Reading followed (paper, Sections "Discussion" and "Future Work": a
stage-specific vector of prefill and decode service deficits; no formula is
given): Eq. (1) split into its prefill part (weighted prefill rate over the
weighted waiting demand) and its decode part (decode rate over the active
demand), each with the one-request floor and the smoothing of Section
"Smoothing, Normalization, and Calibration".
"""
from fractions import Fraction as Fr

import numpy as np

import oracle as O
import tracegen as tg

A_, P_, D_, F_, ADMIT = 0, 1, 2, 3, 0x80


def _prof(M, w_p=0.5, w_q=2.0, alpha=0.5):
    p = np.zeros(M, O.PROFILE_DTYPE)
    p["w_p"], p["w_q"], p["alpha"], p["theta"] = w_p, w_q, alpha, 1.0
    p["tau_crit"], p["tau_surplus"], p["r_min"], p["r_init"] = 0.5, 1.5, 0, 1
    return p


def _trace(rows):
    rows = sorted(rows, key=lambda r: r[0])
    return {"ts": np.array([r[0] for r in rows], np.int64), "model": np.array([r[1] for r in rows], np.uint8),
            "req": np.array([r[2] for r in rows], np.uint32), "type": np.array([r[3] for r in rows], np.uint8),
            "tokens": np.array([r[4] for r in rows], np.uint16)}


def _close(x, exact, what):
    assert np.isfinite(x), f"{what}: {x} vs {float(exact)}"
    assert abs(Fr(float(x)) - exact) <= abs(exact) * Fr(1, 2 ** 50) + Fr(1, 2 ** 1000), f"{what}: {x} vs {float(exact)}"


def pin_hand_trace(o):
    # window 1000 ms, 4 windows; w_p = 1/2, w_q = 2, alpha = 1/2 (all exact in binary)
    # model 0:
    #   req 0: ARRIVE 0 (100-token prompt), PREFILL+ADMIT 100 tokens at 700, DECODE 24 at 800, DECODE 24 at 1200,
    #          FINISH at 1500
    #   req 1: ARRIVE and PREFILL+ADMIT 50 tokens at 1000, DECODE 24 at 1600, DECODE 12 at 2300, FINISH at 2300
    #   req 2: ARRIVE at 3000, never admitted
    # model 1:
    #   req 3: ARRIVE 100, PREFILL+ADMIT 3000 tokens at 200, FINISH at 900 (no output)
    rows = [(0, 0, 0, A_, 100), (700, 0, 0, P_ | ADMIT, 100), (800, 0, 0, D_, 24), (1200, 0, 0, D_, 24),
            (1500, 0, 0, F_, 0),
            (1000, 0, 1, A_, 50), (1000, 0, 1, P_ | ADMIT, 50), (1600, 0, 1, D_, 24), (2300, 0, 1, D_, 12),
            (2300, 0, 1, F_, 0),
            (3000, 0, 2, A_, 10),
            (100, 1, 3, A_, 3000), (200, 1, 3, P_ | ADMIT, 3000), (900, 1, 3, F_, 0)]
    # keep the kind order at equal timestamps (ARRIVE before PREFILL before DECODE before FINISH)
    rows.sort(key=lambda r: (r[0], r[3] & 3))
    ev = _trace(rows)
    prof = _prof(2)
    t = o.tss_trace(ev, 1000, 4000, prof)
    r = o.stage_tss(t, 1000, prof)
    S, fl = r["S"], r["flags"]
    half = Fr(1, 2)
    # model 0, window 0: W on [0, 700) -> W_int 700; A on [700, 1000) -> A_int 300; P 100; D 24
    #   prefill: 1000 * 1/2 * 100 / max(2 * 700, 1000) = 50000 / 1400 = 250/7 (first busy window)
    #   decode:  1000 * 24 / max(300, 1000) = 24 (floor binds)
    sp0, sd0 = Fr(250, 7), Fr(24)
    # window 1: P 50 (req 1, admitted on arrival: W_int 0); A: req 0 on [1000, 1500), req 1 on [1000, 2000)
    #   -> A_int 1500; D 24 + 24 = 48
    #   prefill raw 1000 * 1/2 * 50 / max(0, 1000) = 25 -> S_p = 1/2 * 25 + 1/2 * 250/7 = 425/14
    #   decode raw 48000 / 1500 = 32 (no floor) -> S_d = 1/2 * 32 + 1/2 * 24 = 28
    sp1, sd1 = half * 25 + half * sp0, half * 32 + half * sd0
    # window 2: req 1 active on [2000, 2300): A_int 300, D 12; no prompt tokens, nobody waiting
    #   prefill idle (held); decode raw 12000 / max(300, 1000) = 12 -> S_d = 1/2 * 12 + 1/2 * 28 = 20
    sd2 = half * 12 + half * sd1
    # window 3: req 2 waits on [3000, 4000): W_int 1000, P 0 -> prefill raw 0 / max(2000, 1000) = 0
    #   -> S_p = 1/2 * 0 + 1/2 * 425/14 = 425/28; decode idle (held)
    sp3 = half * 0 + half * sp1
    want0 = [(sp0, sd0, O.P_INIT | O.D_INIT), (sp1, sd1, O.P_INIT | O.D_INIT),
             (sp1, sd2, O.P_IDLE | O.P_INIT | O.D_INIT), (sp3, sd2, O.P_INIT | O.D_IDLE | O.D_INIT)]
    for w, (sp, sd, f) in enumerate(want0):
        _close(S[w, 0, 0], sp, f"model 0 window {w} prefill")
        _close(S[w, 0, 1], sd, f"model 0 window {w} decode")
        assert fl[w, 0] == f, f"model 0 window {w} flags {fl[w, 0]} vs {f}"
    # model 1, window 0: W on [100, 200) -> W_int 100; A on [200, 900) -> A_int 700; P 3000; D 0
    #   prefill: 1000 * 1/2 * 3000 / max(200, 1000) = 1500 (floor binds); decode: 0 / max(700, 1000) = 0
    #   (busy: a request is active); windows 1-3 idle in both stages, values held
    for w in range(4):
        _close(S[w, 1, 0], Fr(1500), f"model 1 window {w} prefill")
        _close(S[w, 1, 1], Fr(0), f"model 1 window {w} decode")
        f = O.P_INIT | O.D_INIT | (0 if w == 0 else O.P_IDLE | O.D_IDLE)
        assert fl[w, 1] == f, f"model 1 window {w} flags {fl[w, 1]} vs {f}"


def _small(w_i, n):
    w = tg.standard(w_i)
    if w.n_traces > 1 or w.duration_ms > 900_000:
        w = w.scaled(n_traces=1, duration_ms=min(w.duration_ms, 900_000))
    return w, w.generate(0, 1, threads=2).trace(0)


def pin_decode_only_reduces_to_base(o):
    """Requests admitted on arrival with empty prompts: no prompt tokens and
    no waiting time anywhere, so Eq. (1) is its decode part."""
    rng = np.random.default_rng(11)
    rows = []
    for rid in range(300):
        m = int(rng.integers(0, 3))
        t = int(rng.integers(0, 500_000))
        rows += [(t, m, rid, A_, 0), (t, m, rid, P_ | ADMIT, 0)]
        n_out = int(rng.integers(1, 6))
        for k in range(n_out):
            t += int(rng.integers(1, 4000))
            rows.append((t, m, rid, D_, int(rng.integers(1, 25))))
        rows.append((t, m, rid, F_, 0))
    rows = [r for r in rows if r[0] < 600_000]
    done = {r[2] for r in rows if r[3] == F_}
    rows = [r for r in rows if r[2] in done]
    rows.sort(key=lambda r: (r[0], r[3] & 3))
    ev = _trace(rows)
    for alpha in (0.3, 0.9, 1.0):
        prof = _prof(3, w_p=0.2, w_q=2.0, alpha=alpha)
        t = o.tss_trace(ev, 1000, 600_000, prof)
        assert (t["P"] == 0).all() and (t["W_int"] == 0).all()
        r = o.stage_tss(t, 1000, prof)
        assert np.array_equal(r["S"][:, :, 1].view(np.uint64), t["S"].view(np.uint64)), "decode share != TSS"
        base_idle = (t["flags"] & O.IDLE) != 0
        assert np.array_equal((r["flags"] & O.D_IDLE) != 0, base_idle)
        assert np.array_equal((r["flags"] & O.D_INIT) != 0, (t["flags"] & O.INIT) != 0)
        assert ((r["flags"] & O.P_IDLE) != 0).all() and ((r["flags"] & O.P_INIT) == 0).all()


def pin_mediant(o):
    """Eq. (1) with both stage denominators above their floors."""
    checked = 0
    for w_i in (0, 1, 3):
        w, ev = _small(w_i, 1)
        prof = O.pack_profiles(w.profile_columns(1))
        t = o.tss_trace(ev, w.window_ms, w.duration_ms, prof)
        W = w.window_ms
        nW, M = t["P"].shape
        for wi in range(nW):
            for m in range(M):
                P, D, Ai, Wi = (int(t[k][wi, m]) for k in ("P", "D", "A_int", "W_int"))
                wp, wq = float(prof["w_p"][m]), float(prof["w_q"][m])
                den_p, den_d = Fr(wq) * Wi, Fr(Ai)
                if den_p < W or den_d < W:
                    continue
                rp = o.stage_raw_prefill(wp, wq, P, Wi, W)
                rd = o.stage_raw_decode(D, Ai, W)
                raw = o.raw_tss(wp, wq, P, D, Ai, Wi, W)
                lo, hi = min(rp, rd), max(rp, rd)
                tol = 4e-16 * max(abs(hi), 1e-300)
                assert lo - tol <= raw <= hi + tol, f"w{wi} m{m}: {raw} not within [{lo}, {hi}]"
                # raw * (den_p + den_d) == rp * den_p + rd * den_d (each side within rounding)
                lhs = Fr(raw) * (den_p + den_d)
                rhs = Fr(rp) * den_p + Fr(rd) * den_d
                assert abs(lhs - rhs) <= (abs(lhs) + 1) * Fr(1, 2 ** 48), f"w{wi} m{m}: mediant identity"
                checked += 1
    assert checked > 100, checked


def pin_special_cases(o):
    # k requests each decoding r tokens/s over the whole window: decode share r
    for k, r in ((1, 48), (3, 96), (5, 20)):
        D = k * r * 2  # over a 2000 ms window
        assert o.stage_raw_decode(D, k * 2000, 2000) == float(r)
    # no waiting: prefill floor of one request
    assert o.stage_raw_prefill(0.25, 3.0, 400, 0, 1000) == 100.0
    # alpha = 1: each share is the raw ratio of its last busy window
    w, ev = _small(1, 1)
    prof = O.pack_profiles(w.profile_columns(1))
    prof["alpha"] = 1.0
    t = o.tss_trace(ev, w.window_ms, w.duration_ms, prof)
    r = o.stage_tss(t, w.window_ms, prof)
    nW, M = t["P"].shape
    for m in range(M):
        lp = ld = None
        for wi in range(nW):
            P, D, Ai, Wi = (int(t[k][wi, m]) for k in ("P", "D", "A_int", "W_int"))
            if P or Wi:
                lp = o.stage_raw_prefill(float(prof["w_p"][m]), float(prof["w_q"][m]), P, Wi, w.window_ms)
            if D or Ai:
                ld = o.stage_raw_decode(D, Ai, w.window_ms)
            if lp is not None:
                assert r["S"][wi, m, 0] == lp
            if ld is not None:
                assert r["S"][wi, m, 1] == ld


def pin_monotone(o):
    rng = np.random.default_rng(3)
    for _ in range(2000):
        W = int(rng.choice([250, 1000, 5000]))
        D, Ai = int(rng.integers(0, 10_000)), int(rng.integers(0, 50_000))
        assert o.stage_raw_decode(D + int(rng.integers(1, 100)), Ai, W) >= o.stage_raw_decode(D, Ai, W)
        P, Wi = int(rng.integers(0, 10_000)), int(rng.integers(0, 50_000))
        wp, wq = float(rng.uniform(0.05, 1)), float(rng.uniform(0.5, 4))
        assert o.stage_raw_prefill(wp, wq, P, Wi + int(rng.integers(1, 5000)), W) <= o.stage_raw_prefill(wp, wq, P, Wi, W)


def pin_bad_arguments_are_rejected(o):
    t = {k: np.zeros((4, 2), np.int64) for k in ("P", "D", "A_int", "W_int")}
    for W in (0, -5):
        try:
            o.stage_tss(t, W, _prof(2))
        except ValueError:
            continue
        raise AssertionError("a non-positive window was accepted")


ALL = [pin_hand_trace, pin_decode_only_reduces_to_base, pin_mediant, pin_special_cases, pin_monotone,
       pin_bad_arguments_are_rejected]
