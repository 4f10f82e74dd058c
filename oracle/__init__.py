"""CPU oracle for TSS evaluation and receiver/donor rebalancing.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  The GPU
library never calls it and shares no code with it.

The arithmetic lives in ``tre_oracle.c`` (plain C, fp64, single thread,
compiled with ``-ffp-contract=off``); this module only builds it and
marshals numpy arrays.  Function-level citations of the paper are in the C
source.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tre_oracle.c")
_SRC_ACT = os.path.join(_HERE, "tre_oracle_act.c")  # control replay with the actuation model
_SRC_CALIB = os.path.join(_HERE, "tre_oracle_calib.c")  # calibration sweep
_SRC_LOOP = os.path.join(_HERE, "tre_oracle_loop.c")  # closed-loop replay
_SRC_STAGE = os.path.join(_HERE, "tre_oracle_stage.c")  # stage-aware service shares
_LIB = os.path.join(_HERE, "libtre_oracle.so")

CFLAGS = ["-O2", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math", "-std=c11"]

RESCUE, REBALANCE, POOL = 1, 2, 0xFF
IDLE, INIT = 1, 2
P_IDLE, P_INIT, D_IDLE, D_INIT = 1, 2, 4, 8  # stage-aware flags

PROFILE_DTYPE = np.dtype([("w_p", "<f8"), ("w_q", "<f8"), ("alpha", "<f8"), ("theta", "<f8"),
                          ("tau_crit", "<f8"), ("tau_surplus", "<f8"), ("r_min", "<i4"),
                          ("r_init", "<i4")])
SCENARIO_DTYPE = np.dtype([("trace", "<u4"), ("max_moves", "<u4"), ("theta_scale", "<f8"),
                           ("tau_crit_override", "<f8")])
MOVE_DTYPE = np.dtype([("window", "<u4"), ("path", "u1"), ("receiver", "u1"), ("donor", "u1"),
                       ("pad", "u1")])
SLO_DTYPE = np.dtype([("ttft_ms", "<f8"), ("tpot_ms", "<f8"), ("e2e_ms", "<f8"), ("attain_q", "<f8"),
                      ("reliability", "<f8")])
FIT_DTYPE = np.dtype([("theta", "<f8"), ("n_cand", "<u4"), ("n_healthy", "<u4"), ("n_above", "<u4"),
                      ("healthy_above", "<u4"), ("concordant", "<u4"), ("discordant", "<u4")])
REQ_DTYPE = np.dtype([("ttft_ms", "<i8"), ("e2e_ms", "<i8"), ("tpot_ms", "<f8"), ("model", "<i4"),
                      ("complete", "u1"), ("has_tpot", "u1"), ("ok", "u1"), ("pad", "u1")])
assert PROFILE_DTYPE.itemsize == 56 and SCENARIO_DTYPE.itemsize == 24 and MOVE_DTYPE.itemsize == 8
assert SLO_DTYPE.itemsize == 40 and FIT_DTYPE.itemsize == 32 and REQ_DTYPE.itemsize == 32
SVC_DTYPE = np.dtype([("prefill_us", "<u4"), ("decode_us", "<u4")])
LOOP_STATS_DTYPE = np.dtype([("n_arrived", "<u4"), ("n_started", "<u4"), ("n_done", "<u4"), ("n_ok", "<u4"),
                             ("e2e_sum", "<i8"), ("e2e_max", "<i8")])
assert SVC_DTYPE.itemsize == 8 and LOOP_STATS_DTYPE.itemsize == 32


def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with gcc (building the checker is not using it).
    The default library also holds the actuation-model replay and the
    calibration sweep; a library built from another base source (the
    pin-strength tests) does not."""
    srcs = [src] + ([_SRC_ACT, _SRC_CALIB, _SRC_LOOP, _SRC_STAGE] if src == _SRC else [])
    stale = not os.path.exists(out) or any(os.path.getmtime(out) < os.path.getmtime(x) for x in srcs)
    if force or stale:
        tmp = f"{out}.{os.getpid()}.tmp"
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, *srcs, "-lm"])
        os.replace(tmp, out)
    return out


class Oracle:
    """ctypes view of one compiled oracle library (the default, or a variant
    compiled from edited source by the pin-strength tests)."""

    def __init__(self, path: str):
        L = ctypes.CDLL(path)
        vp, i64, i32, u32, f64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_double
        L.oracle_raw_tss.restype = f64
        L.oracle_raw_tss.argtypes = [f64, f64, i64, i64, i64, i64, i64]
        L.oracle_smooth.restype = f64
        L.oracle_smooth.argtypes = [f64, f64, f64]
        L.oracle_tss_trace.restype = ctypes.c_int
        L.oracle_tss_trace.argtypes = [vp, vp, vp, vp, i64, i64, i64, i32, vp, vp, vp, vp, vp, vp, vp]
        self.has_admits = hasattr(L, "oracle_check_admits")
        if self.has_admits:
            L.oracle_check_admits.restype = ctypes.c_int
            L.oracle_check_admits.argtypes = [vp, vp, i64, vp, vp]
        self.has_lifecycle = hasattr(L, "oracle_check_lifecycle")
        if self.has_lifecycle:
            L.oracle_check_lifecycle.restype = ctypes.c_int
            L.oracle_check_lifecycle.argtypes = [vp, vp, vp, i64, vp, vp]
        L.oracle_control.restype = ctypes.c_int
        L.oracle_control.argtypes = [i64, i64, i64, i64, i32, i32, vp, vp, vp, vp, vp, u32, vp, vp, vp]
        self.has_act = hasattr(L, "oracle_control_act")
        if self.has_act:
            L.oracle_control_act.restype = ctypes.c_int
            L.oracle_control_act.argtypes = [i64, i64, i64, i64, i32, i32, vp, vp, vp, vp, i64, i64, vp, vp,
                                             vp, u32, vp, vp, vp, vp, vp]
        self.has_calib = hasattr(L, "oracle_calib_requests")
        if self.has_calib:
            L.oracle_calib_requests.restype = i64
            L.oracle_calib_requests.argtypes = [i64, i64, i32, i64, vp, vp, vp, vp, vp, vp, u32, vp, vp, vp]
            L.oracle_calib_fit.restype = ctypes.c_int
            L.oracle_calib_fit.argtypes = [i64, i32, vp, vp, vp, vp, vp, vp]
        self.has_loop = hasattr(L, "oracle_loop")
        if self.has_loop:
            L.oracle_loop.restype = ctypes.c_int
            L.oracle_loop.argtypes = ([i64, i64, i64, i64, i32, i32, vp, vp, vp, vp, i32, i32, i32, i32, vp, vp, vp, vp,
                                       vp, u32, vp, vp, vp, vp, vp, vp, vp, i64, vp, vp, vp, vp])
            L.oracle_loop_act.restype = ctypes.c_int
            L.oracle_loop_act.argtypes = ([i64, i64, i64, i64, i32, i32, vp, vp, vp, vp, i32, i32, i32, i32, vp, vp, vp,
                                           vp, i64, i64, vp, vp, vp, u32, vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, vp,
                                           vp, vp, vp])
        self.has_stage = hasattr(L, "oracle_stage_tss")
        if self.has_stage:
            L.oracle_stage_raw_prefill.restype = f64
            L.oracle_stage_raw_prefill.argtypes = [f64, f64, i64, i64, i64]
            L.oracle_stage_raw_decode.restype = f64
            L.oracle_stage_raw_decode.argtypes = [i64, i64, i64]
            L.oracle_stage_tss.restype = ctypes.c_int
            L.oracle_stage_tss.argtypes = [i64, i32, i64, vp, vp, vp, vp, vp, vp, vp]
        self.L = L
        self.path = path

    # ---------------------------------------------------------------- scalar
    def raw_tss(self, w_p, w_q, P, D, A_int, W_int, window_ms) -> float:
        return self.L.oracle_raw_tss(w_p, w_q, int(P), int(D), int(A_int), int(W_int), int(window_ms))

    def smooth(self, alpha, raw, s_prev) -> float:
        return self.L.oracle_smooth(alpha, raw, s_prev)

    # ----------------------------------------------------------------- trace
    def tss_trace(self, ev: Dict[str, np.ndarray], window_ms: int, duration_ms: int,
                  prof: np.ndarray) -> Dict[str, np.ndarray]:
        """Window tallies and smoothed TSS of one trace; arrays [n_windows][M]."""
        prof = np.ascontiguousarray(prof, dtype=PROFILE_DTYPE)
        M = prof.shape[0]
        nW = duration_ms // window_ms
        ts = np.ascontiguousarray(ev["ts"], np.int64)
        model = np.ascontiguousarray(ev["model"], np.uint8)
        typ = np.ascontiguousarray(ev["type"], np.uint8)
        tok = np.ascontiguousarray(ev["tokens"], np.uint16)
        out = {k: np.zeros((nW, M), np.int64) for k in ("P", "D", "A_int", "W_int")}
        out["S"] = np.zeros((nW, M), np.float64)
        out["flags"] = np.zeros((nW, M), np.uint8)
        rc = self.L.oracle_tss_trace(ts.ctypes.data, model.ctypes.data, typ.ctypes.data, tok.ctypes.data,
                                     ts.shape[0], window_ms, duration_ms, M, prof.ctypes.data,
                                     out["P"].ctypes.data, out["D"].ctypes.data, out["A_int"].ctypes.data,
                                     out["W_int"].ctypes.data, out["S"].ctypes.data, out["flags"].ctypes.data)
        if rc:
            raise ValueError(f"oracle_tss_trace rejected the trace ({rc})")
        return out

    def trace_status(self, ev: Dict[str, np.ndarray], window_ms: int, duration_ms: int, M: int) -> int:
        """The code oracle_tss_trace returns for a trace (0 when it accepts
        it; -2 order, -3 schema, -5 a negative active or waiting count)."""
        nW = duration_ms // window_ms
        prof = np.zeros(M, PROFILE_DTYPE)
        prof["alpha"] = 1.0
        prof["theta"] = 1.0
        ts = np.ascontiguousarray(ev["ts"], np.int64)
        cols = [ts, np.ascontiguousarray(ev["model"], np.uint8), np.ascontiguousarray(ev["type"], np.uint8),
                np.ascontiguousarray(ev["tokens"], np.uint16)]
        outs = [np.zeros((nW, M), np.int64) for _ in range(4)] + [np.zeros((nW, M), np.float64),
                                                                  np.zeros((nW, M), np.uint8)]
        return int(self.L.oracle_tss_trace(*[c.ctypes.data for c in cols], ts.shape[0], window_ms, duration_ms, M,
                                           prof.ctypes.data, *[o.ctypes.data for o in outs]))

    def check_admits(self, ev: Dict[str, np.ndarray]):
        """(0, None) when no request id is admitted twice in the trace, else
        (-6, the smallest such id)."""
        req = np.ascontiguousarray(ev["req"], np.uint32)
        typ = np.ascontiguousarray(ev["type"], np.uint8)
        scratch = np.zeros(max(1, req.shape[0]), np.uint32)
        dup = np.zeros(1, np.uint32)
        rc = int(self.L.oracle_check_admits(req.ctypes.data, typ.ctypes.data, req.shape[0], scratch.ctypes.data,
                                            dup.ctypes.data))
        return rc, (int(dup[0]) if rc else None)

    def check_lifecycle(self, ev: Dict[str, np.ndarray]):
        """(0, None) when every request id of the trace arrives at most once,
        finishes at most once and neither arrives nor decodes at a later
        timestamp than its FINISH; else (-7, the smallest offending id)."""
        req = np.ascontiguousarray(ev["req"], np.uint32)
        typ = np.ascontiguousarray(ev["type"], np.uint8)
        ts = np.ascontiguousarray(ev["ts"], np.int64)
        scratch = np.zeros(max(1, req.shape[0]), np.uint64)
        bad = np.zeros(1, np.uint32)
        rc = int(self.L.oracle_check_lifecycle(req.ctypes.data, typ.ctypes.data, ts.ctypes.data, req.shape[0],
                                               scratch.ctypes.data, bad.ctypes.data))
        return rc, (int(bad[0]) if rc else None)

    def control(self, cfg: Dict[str, int], prof: np.ndarray, S: np.ndarray, flags: np.ndarray,
                sc: np.ndarray, move_cap: Optional[int] = None) -> Dict[str, np.ndarray]:
        """Control replay of one scenario (a 1-element SCENARIO_DTYPE array)."""
        prof = np.ascontiguousarray(prof, dtype=PROFILE_DTYPE)
        sc = np.ascontiguousarray(np.atleast_1d(sc), dtype=SCENARIO_DTYPE)
        M = prof.shape[0]
        nW = cfg["duration_ms"] // cfg["window_ms"]
        if move_cap is None:
            move_cap = max(1, nW * int(sc[0]["max_moves"]))
        S = np.ascontiguousarray(S, np.float64)
        flags = np.ascontiguousarray(flags, np.uint8)
        moves = np.zeros(move_cap, MOVE_DTYPE)
        n_moves = np.zeros(1, np.uint32)
        r_final = np.zeros(M, np.int32)
        r_windows = np.zeros(M, np.int64)
        rc = self.L.oracle_control(cfg["window_ms"], cfg["duration_ms"], cfg["fast_period_ms"],
                                   cfg["slow_period_ms"], M, cfg["budget"], prof.ctypes.data,
                                   S.ctypes.data, flags.ctypes.data, sc.ctypes.data, moves.ctypes.data,
                                   move_cap, n_moves.ctypes.data, r_final.ctypes.data,
                                   r_windows.ctypes.data)
        if rc:
            raise ValueError(f"oracle_control rejected the scenario ({rc})")
        n = int(n_moves[0])
        return {"moves": moves[:min(n, move_cap)].copy(), "n_moves": n, "r_final": r_final,
                "r_windows": r_windows}


    def control_act(self, cfg: Dict[str, int], prof: np.ndarray, S: np.ndarray, flags: np.ndarray,
                    sc: np.ndarray, wake_w: int, sleep_w: int, footprint: Optional[np.ndarray] = None,
                    veto: Optional[np.ndarray] = None, move_cap: Optional[int] = None) -> Dict[str, np.ndarray]:
        """Control replay of one scenario with the actuation model: delays in
        whole windows, footprint [M] GPUs per replica (None: 1), veto
        [n_ticks] uint64 donor-release masks (None: none)."""
        prof = np.ascontiguousarray(prof, dtype=PROFILE_DTYPE)
        sc = np.ascontiguousarray(np.atleast_1d(sc), dtype=SCENARIO_DTYPE)
        M = prof.shape[0]
        nW = cfg["duration_ms"] // cfg["window_ms"]
        if move_cap is None:
            move_cap = max(1, nW * int(sc[0]["max_moves"]))
        S = np.ascontiguousarray(S, np.float64)
        flags = np.ascontiguousarray(flags, np.uint8)
        fp = None if footprint is None else np.ascontiguousarray(footprint, np.int32)
        vt = None if veto is None else np.ascontiguousarray(veto, np.uint64)
        moves = np.zeros(move_cap, MOVE_DTYPE)
        n_moves = np.zeros(1, np.uint32)
        r_final = np.zeros(M, np.int32)
        r_windows = np.zeros(M, np.int64)
        idle = np.zeros(1, np.int64)
        held = np.zeros(M, np.int32)
        rc = self.L.oracle_control_act(
            cfg["window_ms"], cfg["duration_ms"], cfg["fast_period_ms"], cfg["slow_period_ms"], M, cfg["budget"],
            prof.ctypes.data, S.ctypes.data, flags.ctypes.data, sc.ctypes.data, int(wake_w), int(sleep_w),
            None if fp is None else fp.ctypes.data, None if vt is None else vt.ctypes.data, moves.ctypes.data,
            move_cap, n_moves.ctypes.data, r_final.ctypes.data, r_windows.ctypes.data, idle.ctypes.data,
            held.ctypes.data)
        if rc:
            raise ValueError(f"oracle_control_act rejected the scenario ({rc})")
        n = int(n_moves[0])
        return {"moves": moves[:min(n, move_cap)].copy(), "n_moves": n, "r_final": r_final,
                "r_windows": r_windows, "idle_final": int(idle[0]), "held_final": held}


    # ----------------------------------------------------------- closed loop
    def loop(self, cfg: Dict[str, int], prof: np.ndarray, sc: np.ndarray, slo: np.ndarray, svc: np.ndarray,
             reqs: Dict[str, np.ndarray], spr: int = 8, r_cap: int = 16, prefill_chunk: int = 2048,
             decode_chunk: int = 24, move_cap: Optional[int] = None, want_events: bool = False,
             want_tss: bool = False, wake_w: int = 0, sleep_w: int = 0, footprint: Optional[np.ndarray] = None,
             veto: Optional[np.ndarray] = None) -> Dict[str, np.ndarray]:
        """Closed-loop replay of one scenario over one trace's request table
        (arrival_ms, model, prompt, output; model by model, arrivals in
        order within a model). With wake_w / sleep_w (whole windows),
        footprint [M] (GPUs per replica, the budget then in GPUs) or veto
        [n_ticks] (uint64 donor-release masks), the actuation model."""
        prof = np.ascontiguousarray(prof, dtype=PROFILE_DTYPE)
        sc = np.ascontiguousarray(np.atleast_1d(sc), dtype=SCENARIO_DTYPE)
        slo = np.ascontiguousarray(slo, dtype=SLO_DTYPE)
        svc = np.ascontiguousarray(svc, dtype=SVC_DTYPE)
        M = prof.shape[0]
        nW = cfg["duration_ms"] // cfg["window_ms"]
        model = np.asarray(reqs["model"], np.int64)
        assert (np.diff(model) >= 0).all(), "requests must be grouped by model"
        req_off = np.zeros(M + 1, np.int64)
        req_off[1:] = np.cumsum(np.bincount(model, minlength=M)[:M])
        arr = np.ascontiguousarray(reqs["arrival_ms"], np.int64)
        pr = np.ascontiguousarray(reqs["prompt"], np.uint16)
        ou = np.ascontiguousarray(reqs["output"], np.uint16)
        if move_cap is None:
            move_cap = max(1, nW * int(sc[0]["max_moves"]))
        moves = np.zeros(move_cap, MOVE_DTYPE)
        n_moves = np.zeros(1, np.uint32)
        r_final = np.zeros(M, np.int32)
        r_windows = np.zeros(M, np.int64)
        stats = np.zeros(M, LOOP_STATS_DTYPE)
        S = np.zeros((nW, M), np.float64) if want_tss else None
        fl = np.zeros((nW, M), np.uint8) if want_tss else None
        n_ev = np.zeros(1, np.int64)
        cap = 0
        ev = None
        if want_events:
            cap = int(len(arr) * (3 + int(pr.max(initial=0)) // prefill_chunk + int(ou.max(initial=0)) // decode_chunk + 2))
            ev = {"ts": np.zeros(cap, np.int64), "model": np.zeros(cap, np.uint8), "type": np.zeros(cap, np.uint8),
                  "tokens": np.zeros(cap, np.uint16)}
        ptr = lambda a: None if a is None else a.ctypes.data
        act = wake_w or sleep_w or footprint is not None or veto is not None
        idle = np.zeros(1, np.int64)
        held = np.zeros(M, np.int32)
        evp = [ptr(None if ev is None else ev[k]) for k in ("ts", "model", "type", "tokens")]
        common = (cfg["window_ms"], cfg["duration_ms"], cfg["fast_period_ms"], cfg["slow_period_ms"], M, cfg["budget"],
                  prof.ctypes.data, sc.ctypes.data, slo.ctypes.data, svc.ctypes.data, spr, r_cap, prefill_chunk,
                  decode_chunk, req_off.ctypes.data, arr.ctypes.data, pr.ctypes.data, ou.ctypes.data)
        if act:
            fp = None if footprint is None else np.ascontiguousarray(footprint, np.int32)
            vt = None if veto is None else np.ascontiguousarray(veto, np.uint64)
            rc = self.L.oracle_loop_act(*common, int(wake_w), int(sleep_w), ptr(fp), ptr(vt), moves.ctypes.data,
                                        move_cap, n_moves.ctypes.data, r_final.ctypes.data, r_windows.ctypes.data,
                                        stats.ctypes.data, idle.ctypes.data, held.ctypes.data, ptr(S), ptr(fl),
                                        n_ev.ctypes.data, cap, *evp)
        else:
            rc = self.L.oracle_loop(*common, moves.ctypes.data, move_cap, n_moves.ctypes.data, r_final.ctypes.data,
                                    r_windows.ctypes.data, stats.ctypes.data, ptr(S), ptr(fl), n_ev.ctypes.data, cap,
                                    *evp)
        if rc:
            raise ValueError(f"oracle_loop rejected the scenario ({rc})")
        n = int(n_moves[0])
        out = {"moves": moves[:min(n, move_cap)].copy(), "n_moves": n, "r_final": r_final, "r_windows": r_windows,
               "stats": stats, "n_events": int(n_ev[0])}
        if act:
            out["idle_final"], out["held_final"] = int(idle[0]), held
        if want_tss:
            out["S"], out["flags"] = S, fl
        if want_events:
            out["events"] = {k: v[:out["n_events"]] for k, v in ev.items()}
        return out

    # ------------------------------------------------------------ stage-aware
    def stage_tss(self, tallies: Dict[str, np.ndarray], window_ms: int, prof: np.ndarray) -> Dict[str, np.ndarray]:
        """Prefill- and decode-stage smoothed shares of one trace from its
        window tallies (P, D, A_int, W_int, each [n_windows][M]): S
        [n_windows][M][2] (prefill, decode), flags [n_windows][M]."""
        prof = np.ascontiguousarray(prof, dtype=PROFILE_DTYPE)
        cols = [np.ascontiguousarray(tallies[k], np.int64) for k in ("P", "D", "A_int", "W_int")]
        nW, M = cols[0].shape
        S = np.zeros((nW, M, 2), np.float64)
        fl = np.zeros((nW, M), np.uint8)
        rc = self.L.oracle_stage_tss(nW, M, window_ms, prof.ctypes.data, *[c.ctypes.data for c in cols],
                                     S.ctypes.data, fl.ctypes.data)
        if rc:
            raise ValueError("oracle_stage_tss rejected its arguments")
        return {"S": S, "flags": fl}

    def stage_raw_prefill(self, w_p, w_q, P, W_int, window_ms) -> float:
        return self.L.oracle_stage_raw_prefill(w_p, w_q, int(P), int(W_int), int(window_ms))

    def stage_raw_decode(self, D, A_int, window_ms) -> float:
        return self.L.oracle_stage_raw_decode(int(D), int(A_int), int(window_ms))

    # ----------------------------------------------------------- calibration
    def calib_requests(self, ev: Dict[str, np.ndarray], window_ms: int, duration_ms: int, slo: np.ndarray,
                       req_cap: int) -> Dict[str, np.ndarray]:
        """Per-request latencies and per-window SLO attainment of one trace:
        judged / ok [M][n_windows] uint32, reqs [req_cap] REQ_DTYPE, and the
        count of events whose request id is >= req_cap."""
        slo = np.ascontiguousarray(slo, dtype=SLO_DTYPE)
        M = slo.shape[0]
        nW = duration_ms // window_ms if window_ms > 0 else 0  # the C side rejects bad shapes
        cols = [np.ascontiguousarray(ev[k], dt) for k, dt in
                (("ts", np.int64), ("model", np.uint8), ("req", np.uint32), ("type", np.uint8),
                 ("tokens", np.uint16))]
        judged = np.zeros((M, nW), np.uint32)
        ok = np.zeros((M, nW), np.uint32)
        reqs = np.zeros(max(int(req_cap), 1), REQ_DTYPE)
        bad = self.L.oracle_calib_requests(window_ms, duration_ms, M, cols[0].shape[0], *[c.ctypes.data for c in cols],
                                           slo.ctypes.data, int(req_cap), judged.ctypes.data, ok.ctypes.data,
                                           reqs.ctypes.data)
        if bad < 0:
            raise ValueError("oracle_calib_requests rejected the trace")
        return {"judged": judged, "ok": ok, "reqs": reqs[:int(req_cap)], "bad_ids": int(bad)}

    def calib_fit(self, S: np.ndarray, flags: np.ndarray, judged: np.ndarray, ok: np.ndarray,
                  slo: np.ndarray) -> np.ndarray:
        """theta fit per model of one trace: S, flags [n_windows][M]; judged,
        ok [M][n_windows]. Returns FIT_DTYPE [M]."""
        slo = np.ascontiguousarray(slo, dtype=SLO_DTYPE)
        S = np.ascontiguousarray(S, np.float64)
        flags = np.ascontiguousarray(flags, np.uint8)
        judged = np.ascontiguousarray(judged, np.uint32)
        ok = np.ascontiguousarray(ok, np.uint32)
        nW, M = S.shape
        assert flags.shape == (nW, M) and judged.shape == (M, nW) and ok.shape == (M, nW) and slo.shape == (M,)
        fit = np.zeros(M, FIT_DTYPE)
        rc = self.L.oracle_calib_fit(nW, M, S.ctypes.data, flags.ctypes.data, judged.ctypes.data, ok.ctypes.data,
                                     slo.ctypes.data, fit.ctypes.data)
        if rc:
            raise ValueError("oracle_calib_fit rejected its arguments")
        return fit

    def calibrate(self, ev: Dict[str, np.ndarray], window_ms: int, duration_ms: int, prof: np.ndarray,
                  slo: np.ndarray, req_cap: int) -> Dict[str, np.ndarray]:
        """The whole calibration sweep of one trace: TSS, per-request join and
        attainment, then the fit."""
        r = self.tss_trace(ev, window_ms, duration_ms, prof)
        q = self.calib_requests(ev, window_ms, duration_ms, slo, req_cap)
        q["fit"] = self.calib_fit(r["S"], r["flags"], q["judged"], q["ok"], slo)
        q["S"], q["flags"] = r["S"], r["flags"]
        return q


def pack_svc(cols: Dict[str, np.ndarray]) -> np.ndarray:
    n = cols["decode_us"].shape[0]
    a = np.zeros(n, SVC_DTYPE)
    for k in SVC_DTYPE.names:
        a[k] = cols[k]
    return a


def pack_slo(cols: Dict[str, np.ndarray]) -> np.ndarray:
    n = cols["ttft_ms"].shape[0]
    a = np.zeros(n, SLO_DTYPE)
    for k in SLO_DTYPE.names:
        a[k] = cols[k]
    return a


_default: Optional[Oracle] = None


def get() -> Oracle:
    global _default
    if _default is None:
        build(force=False)  # rebuilds when a source is newer
        _default = Oracle(_LIB)
    return _default


def pack_profiles(cols: Dict[str, np.ndarray]) -> np.ndarray:
    n = cols["w_p"].shape[0]
    a = np.zeros(n, PROFILE_DTYPE)
    for k in PROFILE_DTYPE.names:
        a[k] = cols[k]
    return a


def pack_scenarios(cols: Dict[str, np.ndarray]) -> np.ndarray:
    n = cols["trace"].shape[0]
    a = np.zeros(n, SCENARIO_DTYPE)
    for k in SCENARIO_DTYPE.names:
        a[k] = cols[k]
    return a


def run(events, trace_off: np.ndarray, cfg: Dict[str, int], prof_cols: Dict[str, np.ndarray],
        sc_cols: Dict[str, np.ndarray], traces=None, scenarios=None, keep_tss: bool = True):
    """Oracle over a set of traces and scenarios.

    events: dict of host columns; trace_off: CSR offsets (trace i is
    events[off[i]:off[i+1]]); prof_cols: profile columns [n_traces*M];
    sc_cols: scenario columns.  ``traces`` / ``scenarios`` restrict the work
    to subsets (scenarios whose trace is not computed are skipped).
    Returns {"tss": {trace: dict}, "ctl": {scenario: dict}}.
    """
    o = get()
    M = cfg["n_models"]
    prof = pack_profiles(prof_cols)
    sc = pack_scenarios(sc_cols)
    n_traces = len(trace_off) - 1
    traces = range(n_traces) if traces is None else traces
    tss = {}
    for t in traces:
        a, b = int(trace_off[t]), int(trace_off[t + 1])
        ev = {k: events[k][a:b] for k in ("ts", "model", "type", "tokens")}
        tss[t] = o.tss_trace(ev, cfg["window_ms"], cfg["duration_ms"], prof[t * M:(t + 1) * M])
    scenarios = range(sc.shape[0]) if scenarios is None else scenarios
    ctl = {}
    for s in scenarios:
        t = int(sc[s]["trace"])
        if t not in tss:
            continue
        ctl[s] = o.control(cfg, prof[t * M:(t + 1) * M], tss[t]["S"], tss[t]["flags"], sc[s:s + 1])
    if not keep_tss:
        tss = {}
    return {"tss": tss, "ctl": ctl}
