"""Python binding of the C ABI in ``include/tre.h`` (argument marshalling only).

Every step of the replay runs in the HIP kernels of ``libtre.so``; this
module only converts torch tensors (device memory) and the current torch
stream into plain pointers, and raises on a non-OK status.  There is no CPU
fallback: if the library is missing, importing the binding fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtre.so")

TRE_OK, TRE_EINVAL, TRE_EORDER, TRE_ESCHEMA, TRE_ERANGE, TRE_ENOMEM, TRE_EHIP, TRE_ESTATE = range(8)
TRE_VALIDATE = 1
TRE_FLAG_IDLE, TRE_FLAG_INIT = 1, 2
TRE_PATH_RESCUE, TRE_PATH_REBALANCE, TRE_DONOR_POOL = 1, 2, 0xFF
TRE_MAX_MODELS = 64
TRE_NOALLOC_SCRATCH_BYTES = 64 << 20  # include/tre.h

# struct layouts of tre.h
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
REQ_LATENCY_DTYPE = np.dtype([("ttft_ms", "<u4"), ("e2e_ms", "<u4"), ("tpot_ms", "<f8"), ("model", "u1"),
                              ("flags", "u1"), ("pad", "u1", (6,))])
TRE_REQ_ARRIVED, TRE_REQ_COMPLETE, TRE_REQ_TPOT, TRE_REQ_OK = 1, 2, 4, 8
SERVICE_DTYPE = np.dtype([("prefill_us", "<u4"), ("decode_us", "<u4")])
LOOP_STATS_DTYPE = np.dtype([("n_arrived", "<u4"), ("n_started", "<u4"), ("n_done", "<u4"), ("n_ok", "<u4"),
                             ("e2e_sum", "<i8"), ("e2e_max", "<i8")])


class TreError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"TRE status {code}: {msg}")
        self.code = code


class _TraceCfg(ctypes.Structure):
    _fields_ = [("window_ms", ctypes.c_int64), ("duration_ms", ctypes.c_int64),
                ("fast_period_ms", ctypes.c_int64), ("slow_period_ms", ctypes.c_int64),
                ("n_models", ctypes.c_int32), ("budget", ctypes.c_int32)]


class _Info(ctypes.Structure):
    _fields_ = [("n_traces", ctypes.c_uint32), ("n_models", ctypes.c_uint32),
                ("n_events", ctypes.c_int64), ("n_windows", ctypes.c_int64),
                ("n_ticks", ctypes.c_int64)]


class _TssOut(ctypes.Structure):
    _fields_ = [(k, ctypes.c_void_p) for k in
                ("prefill", "decode", "a_int", "w_int", "tss64", "tss32", "flags")]


class _CtlOut(ctypes.Structure):
    _fields_ = [("moves", ctypes.c_void_p), ("move_cap", ctypes.c_uint32),
                ("n_moves", ctypes.c_void_p), ("r_final", ctypes.c_void_p),
                ("r_windows", ctypes.c_void_p)]


class _LoopRequests(ctypes.Structure):
    _fields_ = [(k, ctypes.c_void_p) for k in ("arrival_ms", "prompt", "output", "req_off", "service", "slo")] + \
               [(k, ctypes.c_int32) for k in ("slots_per_replica", "r_cap", "prefill_chunk", "decode_chunk")] + \
               [(k, ctypes.c_uint32) for k in ("max_prompt", "max_output", "max_prefill_us", "max_decode_us",
                                               "max_replicas")]


class _Actuation(ctypes.Structure):
    _fields_ = [("wake_ms", ctypes.c_int64), ("sleep_ms", ctypes.c_int64), ("footprint", ctypes.c_void_p),
                ("veto", ctypes.c_void_p)]


EXPORTS = ["tre_last_error", "tre_load_events", "tre_free_events", "tre_events_info",
           "tre_check_params", "tre_workspace_size", "tre_eval_tss", "tre_rebalance", "tre_sweep",
           "tre_set_timing", "tre_kernel_time", "tre_check_actuation", "tre_rebalance_act", "tre_sweep_act",
           "tre_calib_workspace_size", "tre_calibrate", "tre_loop_workspace_size", "tre_loop", "tre_loop_act",
           "tre_stage_tss", "tre_eval_stage", "tre_sweep_noalloc", "tre_calib_order"]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    vp, u32, i32, sz = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_int, ctypes.c_size_t
    L.tre_last_error.restype = ctypes.c_char_p
    L.tre_last_error.argtypes = []
    L.tre_load_events.restype = i32
    L.tre_load_events.argtypes = [vp, vp, vp, vp, vp, vp, u32, ctypes.POINTER(_TraceCfg), u32, vp,
                                  ctypes.POINTER(ctypes.c_void_p)]
    L.tre_free_events.restype = None
    L.tre_free_events.argtypes = [vp]
    L.tre_events_info.restype = i32
    L.tre_events_info.argtypes = [vp, ctypes.POINTER(_Info)]
    L.tre_check_params.restype = i32
    L.tre_check_params.argtypes = [vp, vp, vp, u32]
    L.tre_workspace_size.restype = i32
    L.tre_workspace_size.argtypes = [vp, u32, ctypes.POINTER(sz)]
    L.tre_eval_tss.restype = i32
    L.tre_eval_tss.argtypes = [vp, vp, ctypes.POINTER(_TssOut), vp]
    L.tre_rebalance.restype = i32
    L.tre_rebalance.argtypes = [vp, vp, vp, vp, vp, u32, ctypes.POINTER(_CtlOut), vp]
    L.tre_sweep.restype = i32
    L.tre_sweep.argtypes = [vp, vp, vp, u32, ctypes.POINTER(_CtlOut), vp, vp, sz, vp]
    L.tre_sweep_noalloc.restype = i32
    L.tre_sweep_noalloc.argtypes = [vp, vp, vp, u32, ctypes.POINTER(_CtlOut), vp, vp]
    L.tre_check_actuation.restype = i32
    L.tre_check_actuation.argtypes = [vp, vp, ctypes.POINTER(_Actuation)]
    L.tre_rebalance_act.restype = i32
    L.tre_rebalance_act.argtypes = [vp, vp, vp, vp, vp, u32, ctypes.POINTER(_Actuation), ctypes.POINTER(_CtlOut), vp]
    L.tre_sweep_act.restype = i32
    L.tre_sweep_act.argtypes = [vp, vp, vp, u32, ctypes.POINTER(_Actuation), ctypes.POINTER(_CtlOut), vp, vp, sz, vp]
    L.tre_calib_workspace_size.restype = i32
    L.tre_calib_workspace_size.argtypes = [vp, u32, ctypes.POINTER(sz)]
    L.tre_calibrate.restype = i32
    L.tre_calibrate.argtypes = [vp, vp, vp, vp, u32, vp, vp, vp, vp, vp, sz, vp]
    L.tre_calib_order.restype = i32
    L.tre_calib_order.argtypes = [vp, vp, vp, vp, vp, vp, vp]
    L.tre_loop_workspace_size.restype = i32
    L.tre_loop_workspace_size.argtypes = [ctypes.POINTER(_TraceCfg), ctypes.POINTER(_LoopRequests), u32,
                                          ctypes.POINTER(sz)]
    L.tre_loop.restype = i32
    L.tre_loop.argtypes = [ctypes.POINTER(_TraceCfg), u32, ctypes.POINTER(_LoopRequests), vp, vp, u32,
                           ctypes.POINTER(_CtlOut), vp, vp, vp, sz, vp]
    L.tre_loop_act.restype = i32
    L.tre_loop_act.argtypes = [ctypes.POINTER(_TraceCfg), u32, ctypes.POINTER(_LoopRequests), vp, vp, u32,
                               ctypes.POINTER(_Actuation), ctypes.POINTER(_CtlOut), vp, vp, vp, sz, vp]
    L.tre_stage_tss.restype = i32
    L.tre_stage_tss.argtypes = [vp, vp, ctypes.POINTER(_TssOut), vp, vp, vp, vp]
    L.tre_eval_stage.restype = i32
    L.tre_eval_stage.argtypes = [vp, vp, vp, vp, vp, vp]
    L.tre_set_timing.restype = i32
    L.tre_set_timing.argtypes = [i32]
    L.tre_kernel_time.restype = i32
    L.tre_kernel_time.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(ctypes.c_uint64)]
    return L


_L = _load()


def _check(rc: int):
    if rc != TRE_OK:
        raise TreError(rc, _L.tre_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("device tensor expected")
    if not t.is_contiguous():
        raise ValueError("contiguous tensor expected")
    return t.data_ptr()


def _table(t: torch.Tensor, n: int, dt: np.dtype, name: str):
    """_ptr of a device table of at least n records of the struct `dt` (the
    library reads n of them through the plain pointer)."""
    have = t.numel() * t.element_size()
    if have < n * dt.itemsize:
        raise ValueError(f"{name}: {have} bytes, {n} records of {dt.itemsize} bytes needed")
    return _ptr(t)


def _prof(ev, prof: torch.Tensor):
    return _table(prof, ev.n_traces * ev.n_models, PROFILE_DTYPE, "profile table")


def _slo(ev, slo: torch.Tensor):
    return _table(slo, ev.n_traces * ev.n_models, SLO_DTYPE, "SLO table")


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream or None


class Events:
    """A loaded trace set (wraps ``tre_events*``); keeps its columns alive."""

    def __init__(self, handle: int, cols: Dict[str, torch.Tensor], cfg: Dict[str, int]):
        self.handle = handle
        self.cols = cols
        self.cfg = dict(cfg)
        info = _Info()
        _check(_L.tre_events_info(handle, ctypes.byref(info)))
        self.n_traces = info.n_traces
        self.n_models = info.n_models
        self.n_events = info.n_events
        self.n_windows = info.n_windows
        self.n_ticks = info.n_ticks

    def close(self):
        if self.handle:
            _L.tre_free_events(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def tre_load_events(ts: torch.Tensor, model: torch.Tensor, req: Optional[torch.Tensor],
                    type: torch.Tensor, tokens: torch.Tensor, trace_off, cfg: Dict[str, int],
                    validate: bool = True, stream=None) -> Events:
    off = np.ascontiguousarray(np.asarray(trace_off, dtype=np.int64))
    c = _TraceCfg(cfg["window_ms"], cfg["duration_ms"], cfg["fast_period_ms"], cfg["slow_period_ms"],
                  cfg["n_models"], cfg["budget"])
    for name, t, dt in (("ts", ts, torch.int64), ("model", model, torch.uint8),
                        ("type", type, torch.uint8), ("tokens", tokens, torch.uint16)):
        if t.dtype != dt:
            raise ValueError(f"{name} must be {dt}")
    h = ctypes.c_void_p()
    _check(_L.tre_load_events(_ptr(ts), _ptr(model), _ptr(req), _ptr(type), _ptr(tokens),
                              off.ctypes.data, len(off) - 1, ctypes.byref(c),
                              TRE_VALIDATE if validate else 0, _stream(stream), ctypes.byref(h)))
    return Events(h.value, {"ts": ts, "model": model, "req": req, "type": type, "tokens": tokens}, cfg)


def pack(cols: Dict[str, np.ndarray], dtype: np.dtype, device="cuda") -> torch.Tensor:
    """Columns -> array of tre.h structs, as a byte tensor on `device`."""
    n = len(next(iter(cols.values())))
    a = np.zeros(n, dtype)
    for k in dtype.names:
        if k in cols:
            a[k] = cols[k]
    return torch.from_numpy(a.view(np.uint8).copy()).to(device)


def unpack_moves(moves: torch.Tensor) -> np.ndarray:
    return moves.cpu().numpy().view(MOVE_DTYPE)


def tre_check_params(ev: Events, prof: torch.Tensor, sc: Optional[torch.Tensor] = None):
    n_sc = 0 if sc is None else sc.numel() // SCENARIO_DTYPE.itemsize
    _check(_L.tre_check_params(ev.handle, _prof(ev, prof), _ptr(sc), n_sc))


def tre_workspace_size(ev: Events, n_scenarios: int) -> int:
    n = ctypes.c_size_t()
    _check(_L.tre_workspace_size(ev.handle, n_scenarios, ctypes.byref(n)))
    return n.value


def tss_outputs(ev: Events, which=("prefill", "decode", "a_int", "w_int", "tss64", "tss32", "flags"),
                device="cuda") -> Dict[str, torch.Tensor]:
    shape = (ev.n_traces, ev.n_windows, ev.n_models)
    dt = {"prefill": torch.int32, "decode": torch.int32, "a_int": torch.int64, "w_int": torch.int64,
          "tss64": torch.float64, "tss32": torch.float32, "flags": torch.uint8}
    return {k: torch.empty(shape, dtype=dt[k], device=device) for k in which}


def tre_eval_tss(ev: Events, prof: torch.Tensor, out: Dict[str, torch.Tensor], stream=None):
    """Fill the given per-cell outputs (prefill/decode are uint32 data in
    int32 tensors)."""
    o = _TssOut(*[_ptr(out.get(k)) for k in ("prefill", "decode", "a_int", "w_int", "tss64", "tss32", "flags")])
    _check(_L.tre_eval_tss(ev.handle, _prof(ev, prof), ctypes.byref(o), _stream(stream)))


STAGE_P_IDLE, STAGE_P_INIT, STAGE_D_IDLE, STAGE_D_INIT = 1, 2, 4, 8


def stage_outputs(ev: Events, which=("stage64", "stage32", "flags"), device="cuda") -> Dict[str, torch.Tensor]:
    """Output tensors of tre_stage_tss: stage64 / stage32 [n_traces][n_windows]
    [n_models][2] (prefill, decode), flags [n_traces][n_windows][n_models]."""
    shape = (ev.n_traces, ev.n_windows, ev.n_models)
    dt = {"stage64": torch.float64, "stage32": torch.float32}
    out = {k: torch.empty(shape + (2,), dtype=dt[k], device=device) for k in which if k in dt}
    if "flags" in which:
        out["flags"] = torch.empty(shape, dtype=torch.uint8, device=device)
    return out


def tre_stage_tss(ev: Events, prof: torch.Tensor, tallies: Dict[str, torch.Tensor], out: Dict[str, torch.Tensor],
                  stream=None):
    """Stage-aware shares from the prefill / decode / a_int / w_int outputs of
    tre_eval_tss; fills the given outputs."""
    t = _TssOut(*[_ptr(tallies.get(k)) for k in ("prefill", "decode", "a_int", "w_int")], None, None, None)
    _check(_L.tre_stage_tss(ev.handle, _prof(ev, prof), ctypes.byref(t), _ptr(out.get("stage64")),
                            _ptr(out.get("stage32")), _ptr(out.get("flags")), _stream(stream)))


def tre_eval_stage(ev: Events, prof: torch.Tensor, out: Dict[str, torch.Tensor], stream=None):
    """Stage-aware shares straight from the events (one pass, no tallies in
    HBM); fills the given outputs of stage_outputs()."""
    _check(_L.tre_eval_stage(ev.handle, _prof(ev, prof), _ptr(out.get("stage64")), _ptr(out.get("stage32")),
                             _ptr(out.get("flags")), _stream(stream)))


def ctl_outputs(ev: Events, n_scenarios: int, move_cap: int, device="cuda") -> Dict[str, torch.Tensor]:
    M = ev.n_models
    return {"moves": torch.zeros(max(1, n_scenarios * move_cap) * MOVE_DTYPE.itemsize, dtype=torch.uint8, device=device),
            "move_cap": move_cap,
            "n_moves": torch.zeros(max(1, n_scenarios), dtype=torch.int32, device=device),
            "r_final": torch.zeros((max(1, n_scenarios), M), dtype=torch.int32, device=device),
            "r_windows": torch.zeros((max(1, n_scenarios), M), dtype=torch.int64, device=device)}


def _ctl(out) -> _CtlOut:
    return _CtlOut(_ptr(out["moves"]), int(out["move_cap"]), _ptr(out["n_moves"]), _ptr(out["r_final"]),
                   _ptr(out["r_windows"]))


def tre_rebalance(ev: Events, prof: torch.Tensor, tss64: torch.Tensor, flags: torch.Tensor,
                  sc: torch.Tensor, out: Dict[str, torch.Tensor], stream=None):
    n_sc = sc.numel() // SCENARIO_DTYPE.itemsize
    o = _ctl(out)
    _check(_L.tre_rebalance(ev.handle, _prof(ev, prof), _ptr(tss64), _ptr(flags), _ptr(sc), n_sc,
                            ctypes.byref(o), _stream(stream)))


def tre_sweep(ev: Events, prof: torch.Tensor, sc: torch.Tensor, out: Dict[str, torch.Tensor],
              ws: torch.Tensor, tss32: Optional[torch.Tensor] = None, stream=None):
    n_sc = sc.numel() // SCENARIO_DTYPE.itemsize
    o = _ctl(out)
    _check(_L.tre_sweep(ev.handle, _prof(ev, prof), _ptr(sc), n_sc, ctypes.byref(o), _ptr(tss32), _ptr(ws),
                        ws.numel() * ws.element_size(), _stream(stream)))


def tre_sweep_noalloc(ev: Events, prof: torch.Tensor, sc: torch.Tensor, out: Dict[str, torch.Tensor],
                      tss32: Optional[torch.Tensor] = None, stream=None):
    """tre_sweep with its scratch in the library's static device array."""
    n_sc = sc.numel() // SCENARIO_DTYPE.itemsize
    o = _ctl(out)
    _check(_L.tre_sweep_noalloc(ev.handle, _prof(ev, prof), _ptr(sc), n_sc, ctypes.byref(o), _ptr(tss32),
                                _stream(stream)))


def actuation(wake_ms: int, sleep_ms: int, footprint: Optional[torch.Tensor] = None,
              veto: Optional[torch.Tensor] = None) -> _Actuation:
    """The actuation model of include/tre.h: delays in ms; footprint (int32
    [n_traces][n_models]) and veto (uint64 / int64 [n_traces][n_ticks]) are
    device tensors or None. Keep the tensors alive while the model is used."""
    for t, name in ((footprint, "footprint"), (veto, "veto")):
        if t is not None and not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    return _Actuation(int(wake_ms), int(sleep_ms), _ptr(footprint), _ptr(veto))


def tre_check_actuation(ev: Events, prof: torch.Tensor, act: _Actuation):
    _check(_L.tre_check_actuation(ev.handle, _prof(ev, prof), ctypes.byref(act)))


def tre_rebalance_act(ev: Events, prof: torch.Tensor, tss64: torch.Tensor, flags: torch.Tensor,
                      sc: torch.Tensor, act: _Actuation, out: Dict[str, torch.Tensor], stream=None):
    n_sc = sc.numel() // SCENARIO_DTYPE.itemsize
    o = _ctl(out)
    _check(_L.tre_rebalance_act(ev.handle, _prof(ev, prof), _ptr(tss64), _ptr(flags), _ptr(sc), n_sc,
                                ctypes.byref(act), ctypes.byref(o), _stream(stream)))


def tre_sweep_act(ev: Events, prof: torch.Tensor, sc: torch.Tensor, act: _Actuation, out: Dict[str, torch.Tensor],
                  ws: torch.Tensor, tss32: Optional[torch.Tensor] = None, stream=None):
    n_sc = sc.numel() // SCENARIO_DTYPE.itemsize
    o = _ctl(out)
    _check(_L.tre_sweep_act(ev.handle, _prof(ev, prof), _ptr(sc), n_sc, ctypes.byref(act), ctypes.byref(o), _ptr(tss32),
                            _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def tre_calib_workspace_size(ev: Events, req_cap: int) -> int:
    n = ctypes.c_size_t()
    _check(_L.tre_calib_workspace_size(ev.handle, int(req_cap), ctypes.byref(n)))
    return n.value


def calib_outputs(ev: Events, req_cap: int, with_reqs: bool = False, device="cuda") -> Dict[str, torch.Tensor]:
    """Output tensors of tre_calibrate: counts [n_traces][n_models][n_windows]
    (int32 holding judged << 16 | ok), fit and optional per-request records
    as byte tensors (unpack with unpack_fit / unpack_reqs), the id counter and
    the workspace."""
    out = {"counts": torch.empty((ev.n_traces, ev.n_models, ev.n_windows), dtype=torch.int32, device=device),
           "fit": torch.empty(ev.n_traces * ev.n_models * FIT_DTYPE.itemsize, dtype=torch.uint8, device=device),
           "n_bad": torch.empty(1, dtype=torch.int64, device=device),
           "ws": torch.empty(tre_calib_workspace_size(ev, req_cap), dtype=torch.uint8, device=device),
           "req_cap": int(req_cap)}
    out["reqs"] = (torch.empty(ev.n_traces * int(req_cap) * REQ_LATENCY_DTYPE.itemsize, dtype=torch.uint8,
                               device=device) if with_reqs else None)
    return out


def tre_calibrate(ev: Events, slo: torch.Tensor, tss64: torch.Tensor, flags: torch.Tensor,
                  out: Dict[str, torch.Tensor], stream=None):
    ws = out["ws"]
    _check(_L.tre_calibrate(ev.handle, _slo(ev, slo), _ptr(tss64), _ptr(flags), int(out["req_cap"]), _ptr(out["counts"]),
                            _ptr(out["fit"]), _ptr(out.get("reqs")), _ptr(out.get("n_bad")), _ptr(ws),
                            ws.numel() * ws.element_size(), _stream(stream)))


def tre_calib_order(ev: Events, slo: torch.Tensor, tss64: torch.Tensor, flags: torch.Tensor,
                    out: Dict[str, torch.Tensor], stream=None):
    """The fits again with the ordering counts, from tre_calibrate's counts."""
    _check(_L.tre_calib_order(ev.handle, _slo(ev, slo), _ptr(tss64), _ptr(flags), _ptr(out["counts"]), _ptr(out["fit"]),
                              _stream(stream)))


def calib_fallback_traces(ev: Events, out: Dict[str, torch.Tensor]):
    """(traces the last tre_calibrate on `out` redid with the larger stream
    table, traces it redid on the chunked path): the uint32 counts that
    open the workspace's two lists; synchronises."""
    lb = ((4 + 4 * ev.n_traces) + 255) & ~255
    w = out["ws"][256:256 + 2 * lb].cpu().numpy()
    return int(w[0:4].view(np.uint32)[0]), int(w[lb:lb + 4].view(np.uint32)[0])


def unpack_fit(fit: torch.Tensor) -> np.ndarray:
    return fit.cpu().numpy().view(FIT_DTYPE)


def unpack_reqs(reqs: torch.Tensor) -> np.ndarray:
    return reqs.cpu().numpy().view(REQ_LATENCY_DTYPE)


def _cfg(cfg: Dict[str, int]) -> _TraceCfg:
    return _TraceCfg(cfg["window_ms"], cfg["duration_ms"], cfg["fast_period_ms"], cfg["slow_period_ms"],
                     cfg["n_models"], cfg["budget"])


def loop_requests(tables, n_models: int, service: np.ndarray, slo: np.ndarray, slots_per_replica: int = 8,
                  r_cap: int = 16, prefill_chunk: int = 2048, decode_chunk: int = 24, max_replicas: int = 0,
                  device="cuda"):
    """Device request tables of tre_loop from per-trace host tables
    (arrival_ms, model, prompt, output; grouped by model, arrivals in order
    within a model). max_replicas: a declared bound on the replicas holding
    slots at once in one scenario (0: none). Returns (struct, tensors); keep
    the tensors alive."""
    counts = []
    for tb in tables:
        m = np.asarray(tb["model"], np.int64)
        assert (np.diff(m) >= 0).all(), "requests must be grouped by model"
        counts.append(np.bincount(m, minlength=n_models)[:n_models])
    off = np.zeros(len(tables) * n_models + 1, np.int64)
    off[1:] = np.cumsum(np.concatenate(counts) if counts else np.zeros(0, np.int64))
    cat = lambda k, dt: np.concatenate([np.asarray(tb[k], dt) for tb in tables]) if tables else np.zeros(0, dt)
    host = {"arrival_ms": cat("arrival_ms", np.int64), "prompt": cat("prompt", np.uint16),
            "output": cat("output", np.uint16)}
    tens = {k: torch.from_numpy(np.concatenate([v, np.zeros(1, v.dtype)])).to(device) for k, v in host.items()}
    tens["req_off"] = torch.from_numpy(off).to(device)
    svc = np.ascontiguousarray(service, SERVICE_DTYPE)
    tens["service"] = torch.from_numpy(svc.view(np.uint8).copy()).to(device)
    tens["slo"] = torch.from_numpy(np.ascontiguousarray(slo, SLO_DTYPE).view(np.uint8).copy()).to(device)
    rq = _LoopRequests(_ptr(tens["arrival_ms"]), _ptr(tens["prompt"]), _ptr(tens["output"]), _ptr(tens["req_off"]),
                       _ptr(tens["service"]), _ptr(tens["slo"]), slots_per_replica, r_cap, prefill_chunk,
                       decode_chunk, int(host["prompt"].max(initial=1)), int(host["output"].max(initial=1)),
                       int(svc["prefill_us"].max(initial=0)), int(svc["decode_us"].max(initial=0)),
                       int(max_replicas))
    return rq, tens


def tre_loop_workspace_size(cfg: Dict[str, int], rq: _LoopRequests, n_scenarios: int) -> int:
    n = ctypes.c_size_t()
    c = _cfg(cfg)
    _check(_L.tre_loop_workspace_size(ctypes.byref(c), ctypes.byref(rq), n_scenarios, ctypes.byref(n)))
    return n.value


def tre_loop(cfg: Dict[str, int], n_traces: int, rq: _LoopRequests, prof: torch.Tensor, sc: torch.Tensor,
             out: Dict[str, torch.Tensor], stats: torch.Tensor, ws: torch.Tensor,
             tss64: Optional[torch.Tensor] = None, stream=None):
    n_sc = sc.numel() // SCENARIO_DTYPE.itemsize
    c = _cfg(cfg)
    o = _ctl(out)
    prof_p = _table(prof, n_traces * cfg["n_models"], PROFILE_DTYPE, "profile table")
    _check(_L.tre_loop(ctypes.byref(c), n_traces, ctypes.byref(rq), prof_p, _ptr(sc), n_sc, ctypes.byref(o),
                       _ptr(stats), _ptr(tss64), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def tre_loop_act(cfg: Dict[str, int], n_traces: int, rq: _LoopRequests, prof: torch.Tensor, sc: torch.Tensor,
                 act: _Actuation, out: Dict[str, torch.Tensor], stats: torch.Tensor, ws: torch.Tensor,
                 tss64: Optional[torch.Tensor] = None, stream=None):
    """tre_loop with the actuation model (see actuation(); the budget in
    cfg then counts GPUs)."""
    n_sc = sc.numel() // SCENARIO_DTYPE.itemsize
    c = _cfg(cfg)
    o = _ctl(out)
    prof_p = _table(prof, n_traces * cfg["n_models"], PROFILE_DTYPE, "profile table")
    _check(_L.tre_loop_act(ctypes.byref(c), n_traces, ctypes.byref(rq), prof_p, _ptr(sc), n_sc, ctypes.byref(act),
                           ctypes.byref(o), _ptr(stats), _ptr(tss64), _ptr(ws), ws.numel() * ws.element_size(),
                           _stream(stream)))


def tre_set_timing(enable: bool):
    _check(_L.tre_set_timing(1 if enable else 0))


def tre_kernel_time(kernel: str):
    ms, n = ctypes.c_double(), ctypes.c_uint64()
    _check(_L.tre_kernel_time(kernel.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
