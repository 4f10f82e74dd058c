#!/usr/bin/env python3
"""Throughput of the TSS + rebalancing replay on one MI355X.

One step = one ``tre_sweep`` call over the whole resident workload: stream
every event column from HBM, per-(trace, model, window) tallies, carry scan,
Eq. (1) TSS + smoothing, then per scenario Eq. (2), regions, cadence and the
bounded receiver/donor moves.  Events are generated on the host (seeded),
copied to HBM and validated before the timed region; the timed region only
contains the sweeps.

Prints ONE JSON line (rank 0).  ``value`` is request-events per second
(sum over scenarios of the events of that scenario's trace, per second of
sweep time).  ``roofline`` describes the dominant kernel (``tss_stream``):
algorithmic bytes per launch = 12 bytes per physical event (ts 8 + model 1 +
type 1 + tokens 2; the request-id column is never read) divided by the
kernel's mean launch time measured with HIP events on its stream.
``cpu_baseline`` times the CPU oracle (one trace per call, on a pool of
host threads) on a bounded sample of the same traces and checks the GPU's
decisions on that sample.

``--actuation`` replays the same workload under the actuation model
(``tre_sweep_act``): the paper's measured wake and sleep times (1.31 s and
1.87 s, rounded up to whole windows), footprints of 1 or 2 GPUs per replica
drawn from a fixed seed with the GPU budget set to the largest initial
footprint sum plus 8, and donor-release vetoes on 10% of the ticks; the CPU
leg then runs the oracle's actuation replay. With ``--loop`` it replays the
closed loop (``tre_loop_act``) with footprints by model class (7B 1, 13B 1,
34B 2, 70B 4 GPUs per replica), 8 spare GPUs and the replica bound that
follows, declared so that the slot pool is sized for it.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOADS = {"tiny": 0, "bursty": 1, "sweep": 2, "diverse": 3, "stress": 4}
HBM_PEAK_GBS = 8000.0
ALG_BYTES_PER_EVENT = 12
CPU_EVENT_BUDGET = 3_000_000_000
# Oracle threads: the CPU share of one GPU on the measurement hosts (their
# rules cap a one-GPU job's worker pools at 16 whatever the host shows);
# cpu_baseline reports these threads as "cores" and the host's own CPU
# count and model beside them.
CPU_WORKERS = 16
ACT_WAKE_MS, ACT_SLEEP_MS = 1310, 1870  # measured reactivation and sleep times
ACT_SEED = 2609
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "tss_stream_traffic.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2609_29160_amd", "csrc", "tre.hip")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def host_cpu():
    """The host's CPU model (from /proc/cpuinfo), its logical CPUs and the
    CPUs this process may run on."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = None
    return {"cpu_model": model, "host_logical_cpus": os.cpu_count(), "affinity_cpus": affinity}


def kernel_sha(src: str = None) -> str:
    return hashlib.sha256(open(src or KERNEL_SRC, "rb").read()).hexdigest()[:16]


def loop_traffic_for(workload_name: str, key: str = "loop_replay"):
    """HBM bytes per loop_replay launch (key "loop_replay_act": the
    actuation instantiation) from committed counters taken on this kernel
    source and workload; else None."""
    try:
        t = json.load(open(os.path.join(ROOT, "profiles", "loop_traffic.json")))
    except (OSError, ValueError):
        return None
    src = os.path.join(ROOT, "paper_2609_29160_amd", "csrc", "loop.hip")
    if t.get("kernel_sha") != kernel_sha(src) or t.get("workload") != workload_name:
        return None
    return t.get("traffic_bytes_per_launch", {}).get(key)


def traffic_for(workload_name: str, events: int):
    """HBM bytes per tss_stream launch from committed rocprofv3 counters, if
    they were taken on this kernel source and workload; else None."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if t.get("kernel_sha") != kernel_sha() or t.get("workload") != workload_name or t.get("events") != events:
        return None
    return t.get("bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="stress", choices=sorted(WORKLOADS))
    ap.add_argument("--traces", type=int, default=None, help="use only the first N traces")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="traces timed on the CPU oracle (default: the leading traces "
                         "within 3e9 events)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle leg")
    ap.add_argument("--emit-tss", action="store_true", help="also write per-window fp32 TSS")
    ap.add_argument("--threads", type=int, default=None)
    ap.add_argument("--actuation", action="store_true",
                    help="wake/sleep delays, 1-2 GPU footprints and vetoes (tre_sweep_act; with --loop, "
                         "tre_loop_act)")
    ap.add_argument("--loop", action="store_true",
                    help="time the closed-loop replay (tre_loop) over the workload's request tables instead")
    ap.add_argument("--loop-cpu-scenarios", type=int, default=16,
                    help="scenarios replayed by the oracle in the --loop CPU leg")
    ap.add_argument("--stage", action="store_true",
                    help="time the stage-aware shares (tre_eval_stage, one pass; the two-pass path beside it) instead")
    ap.add_argument("--calibrate", action="store_true",
                    help="time the calibration sweep (tre_eval_tss + tre_calibrate) instead")
    ap.add_argument("--copy-calib-gb", type=float, default=0.0,
                    help="after the run, copy this many GB device-to-device (counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(traces and scenarios would shard across GPUs with no exchange)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import tracegen as tg
    from paper_2609_29160_amd import device, tre

    torch.cuda.set_device(0)
    w = tg.standard(WORKLOADS[args.workload])
    if args.traces:
        n = min(args.traces, w.n_traces)
        w = w.scaled(n_traces=n, n_scenarios=n if (w.n_scenarios and w.scenario_trace == "identity") else w.n_scenarios)
    sc_cols = w.scenario_columns()
    n_sc = len(sc_cols["trace"])

    if args.loop:
        return loop_main(args, w, tre, torch, np)
    t0 = time.time()
    dt = device.upload(w, threads=args.threads, log=log)
    log(f"resident: {dt.n_events} events, {dt.stored_bytes / 1e9:.1f} GB stored ({time.time() - t0:.1f} s)")
    if args.calibrate:
        return calibrate_main(args, w, dt, device, tre, torch, np)
    if args.stage:
        return stage_main(args, w, dt, device, tre, torch, np)
    act_in = actuation_inputs(w) if args.actuation else None
    ev = device.load(dt, validate=True, budget=None if act_in is None else act_in["budget"])
    prof = device.profiles(w)
    act = None
    if act_in is not None:
        act_in["veto"] = actuation_vetoes(w, ev.n_ticks)
        act_in["g_dev"] = torch.from_numpy(act_in["g"]).cuda()
        act_in["veto_dev"] = torch.from_numpy(act_in["veto"].view(np.int64)).cuda()
        act = tre.actuation(ACT_WAKE_MS, ACT_SLEEP_MS, act_in["g_dev"], act_in["veto_dev"])
        tre.tre_check_actuation(ev, prof, act)
    sc = device.scenarios(sc_cols)
    tre.tre_check_params(ev, prof, sc)
    max_k = int(np.max(sc_cols["max_moves"]))
    move_cap = max(1, ev.n_ticks * max_k)
    out = tre.ctl_outputs(ev, n_sc, move_cap)
    ws = torch.empty(tre.tre_workspace_size(ev, n_sc), dtype=torch.uint8, device="cuda")
    tss32 = None
    if args.emit_tss:
        tss32 = torch.empty((ev.n_traces, ev.n_windows, ev.n_models), dtype=torch.float32, device="cuda")
    counts = dt.counts
    logical = int(sum(int(counts[int(t)]) for t in sc_cols["trace"]))
    log(f"{ev.n_traces} traces, {n_sc} scenarios, {ev.n_windows} windows, {ev.n_ticks} ticks, "
        f"{logical} logical events")

    def sweep():
        if act is None:
            tre.tre_sweep(ev, prof, sc, out, ws, tss32=tss32)
        else:
            tre.tre_sweep_act(ev, prof, sc, act, out, ws, tss32=tss32)

    for _ in range(args.warmup):
        sweep()
    torch.cuda.synchronize()
    log("warmup done")

    stream = torch.cuda.current_stream()
    tre.tre_set_timing(True)
    tre.tre_kernel_time("tss_stream")
    tre.tre_kernel_time("rebalance")
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        sweep()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    tre.tre_set_timing(False)
    step_ms = e0.elapsed_time(e1) / args.steps
    k_ms, k_n = tre.tre_kernel_time("tss_stream")
    r_ms, r_n = tre.tre_kernel_time("rebalance")
    stream_ms = k_ms / max(k_n, 1)
    reb_ms = r_ms / max(r_n, 1)
    log(f"step {step_ms:.3f} ms (wall {1e3 * wall / args.steps:.3f} ms); tss_stream {stream_ms:.3f} ms, "
        f"rebalance {reb_ms:.3f} ms")

    value = logical / (step_ms / 1e3)
    alg_bytes = ALG_BYTES_PER_EVENT * dt.n_events
    achieved = alg_bytes / (stream_ms / 1e3) / 1e9
    traffic = traffic_for(w.name, dt.n_events)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": "tss_stream", "kernel_ms": round(stream_ms, 4),
                "alg_bytes_per_launch": alg_bytes}

    stream_read = flat_read_rate(dt.cols["ts"], torch)
    log(f"flat read of the ts column: {stream_read['gbs']} GB/s")
    cpu = None
    parity = None
    if not args.no_cpu:
        # the leading traces whose events fit the oracle's budget (about 30 s
        # of host CPU time at ~1e8 events/s per thread), or --cpu-sample traces
        if args.cpu_sample:
            n_s = min(args.cpu_sample, w.n_traces)
        else:
            n_s = max(1, int(np.searchsorted(np.cumsum(dt.counts), CPU_EVENT_BUDGET, side="right")))
        cpu, parity = cpu_leg(w, list(range(n_s)), sc_cols, out, move_cap, tre, args.threads, act_in)

    result = {
        "metric": "request-events/sec through TSS+rebalance (1 GPU); achieved HBM GB/s vs peak",
        "value": round(value, 1),
        "unit": "request-events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic (seeded generator; the paper's traces are not available)",
        "config": {"workload": w.name, "traces": ev.n_traces, "scenarios": n_sc, "models": ev.n_models,
                   "window_ms": w.window_ms, "duration_s": w.duration_ms // 1000,
                   "events": dt.n_events, "logical_events": logical,
                   "stored_gb": round(dt.stored_bytes / 1e9, 2), "emit_tss": bool(args.emit_tss),
                   "actuation": None if act_in is None else
                   {"wake_ms": ACT_WAKE_MS, "sleep_ms": ACT_SLEEP_MS, "footprint_gpus": "1-2, seeded",
                    "budget_gpus": act_in["budget"], "veto_tick_fraction": 0.1}},
        "roofline": roofline,
        "stream_read": stream_read,
        "cpu_baseline": cpu,
        "parity": parity,
        "rebalance_ms": round(reb_ms, 4),
    }
    print(json.dumps(result), flush=True)

    if args.copy_calib_gb > 0:
        copy_calibration(args.copy_calib_gb, torch)
    ev.close()


CALIB_KERNELS = ("tss_stream", "calib_fill", "calib_stream", "calib_fallback", "calib_fit")


def loop_main(args, w, tre, torch, np):
    """One step = tre_loop over every scenario of the workload: each model's
    requests served on its replicas' slots, the controller's moves changing
    them, the TSS from the events this service produces. The request tables
    (the same arrivals and lengths as the workload's traces) are generated
    on host threads and copied to HBM before the timed region. Algorithmic
    bytes per launch: 12 per request of each scenario's trace (arrival,
    prompt and output lengths read once); the kernel is bound by each
    scenario's sequential chain of windows, not by bytes."""
    from concurrent.futures import ThreadPoolExecutor

    T, M = w.n_traces, w.n_models
    n_workers = max(1, min(CPU_WORKERS, os.cpu_count() or 1))
    t0 = time.time()
    with ThreadPoolExecutor(max_workers=n_workers) as pool:
        tables = list(pool.map(w.requests, range(T)))
    svc = np.zeros(T * M, tre.SERVICE_DTYPE)
    for k, v in w.service_columns().items():
        svc[k] = v
    slo = np.zeros(T * M, tre.SLO_DTYPE)
    for k, v in w.slo_columns().items():
        slo[k] = v
    n_req_trace = np.array([len(tb["arrival_ms"]) for tb in tables], np.int64)
    log(f"request tables: {int(n_req_trace.sum())} requests in {T} traces ({time.time() - t0:.1f} s)")
    cfg = w.trace_cfg()
    from paper_2609_29160_amd import device
    prof = device.profiles(w)
    sc_cols = w.scenario_columns()
    n_sc = len(sc_cols["trace"])
    sc = tre.pack(sc_cols, tre.SCENARIO_DTYPE)
    nW = w.n_windows
    n_ticks = sum(1 for x in range(nW) if ((x + 1) * w.window_ms) % cfg["fast_period_ms"] == 0
                  or ((x + 1) * w.window_ms) % cfg["slow_period_ms"] == 0)
    move_cap = max(1, n_ticks * int(np.max(sc_cols["max_moves"])))

    class _Shape:
        n_models = M

    act_in = None
    if args.actuation:
        act_in = loop_actuation_inputs(w)
        act_in["veto"] = actuation_vetoes(w, n_ticks)
        act_in["g_dev"] = torch.from_numpy(act_in["g"]).cuda()
        act_in["veto_dev"] = torch.from_numpy(act_in["veto"].view(np.int64)).cuda()
        cfg = dict(cfg, budget=act_in["budget"])
        act = tre.actuation(ACT_WAKE_MS, ACT_SLEEP_MS, act_in["g_dev"], act_in["veto_dev"])
    rq, keep = tre.loop_requests(tables, M, svc, slo, max_replicas=0 if act_in is None else act_in["max_replicas"])

    def replay():
        if act_in is None:
            tre.tre_loop(cfg, T, rq, prof, sc, out, stats, ws)
        else:
            tre.tre_loop_act(cfg, T, rq, prof, sc, act, out, stats, ws)

    out = tre.ctl_outputs(_Shape(), n_sc, move_cap)
    stats = torch.zeros(n_sc * M * tre.LOOP_STATS_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    ws = torch.empty(tre.tre_loop_workspace_size(cfg, rq, n_sc), dtype=torch.uint8, device="cuda")
    log(f"closed loop: {n_sc} scenarios, workspace {ws.numel() / 1e9:.2f} GB"
        + ("" if act_in is None else f", actuation model (GPU budget {act_in['budget']})"))
    for _ in range(args.warmup):
        replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    tre.tre_set_timing(True)
    tre.tre_kernel_time("loop_replay")
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        replay()
    e1.record(stream)
    torch.cuda.synchronize()
    tre.tre_set_timing(False)
    step_ms = e0.elapsed_time(e1) / args.steps
    k_ms, k_n = tre.tre_kernel_time("loop_replay")
    kern_ms = k_ms / max(k_n, 1)
    overflow = int(ws[:8].cpu().numpy().view(np.uint64)[0])
    logical = int(sum(int(n_req_trace[int(t)]) for t in sc_cols["trace"]))
    alg = 12 * logical
    log(f"step {step_ms:.3f} ms; loop_replay {kern_ms:.3f} ms; events beyond the ring {overflow}")
    cpu = parity = None
    if not args.no_cpu:
        cpu, parity = loop_cpu_leg(w, tables, sc_cols, out, stats, move_cap, args.loop_cpu_scenarios, n_workers, tre,
                                   act_in)
    if args.copy_calib_gb > 0:
        del ws, out, stats, rq, keep
        torch.cuda.empty_cache()
        copy_calibration(args.copy_calib_gb, torch)
    result = {
        "metric": "requests/sec through the closed-loop replay (1 GPU)",
        "value": round(logical / (step_ms / 1e3), 1),
        "unit": "requests/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic (seeded generator; the paper's traces are not available)",
        "config": {"workload": w.name, "traces": T, "scenarios": n_sc, "models": M, "window_ms": w.window_ms,
                   "duration_s": w.duration_ms // 1000, "requests": int(n_req_trace.sum()), "logical_requests": logical,
                   "slots_per_replica": 8, "r_cap": 16, "mode": "closed loop",
                   "actuation": None if act_in is None else
                   {"wake_ms": ACT_WAKE_MS, "sleep_ms": ACT_SLEEP_MS,
                    "footprint_gpus": "by model class: " + ", ".join(f"{k} {v}" for k, v in CLASS_GPUS.items()),
                    "gpu_budget": act_in["budget"], "max_replicas": act_in["max_replicas"], "veto_ticks": "10%"}},
        "roofline": {"bound": "hbm", "achieved": round(alg / (kern_ms / 1e3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(alg / (kern_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": loop_traffic_for(w.name, "loop_replay" if act_in is None else "loop_replay_act")
                     if T == 4096 else None, "kernel": "loop_replay",
                     "kernel_ms": round(kern_ms, 4), "alg_bytes_per_launch": alg,
                     "note": "latency-bound: each scenario is a sequential chain of windows; HBM is not "
                             "the limit (profiles/loop_replay_sq_counters_stress.md)"},
        "events_beyond_ring": overflow,
        "cpu_baseline": cpu, "parity": parity,
    }
    print(json.dumps(result), flush=True)


def loop_cpu_leg(w, tables, sc_cols, out, stats, move_cap, n_sample, n_workers, tre, act_in=None):
    """The oracle's closed-loop replay of the first n_sample scenarios on a
    pool of host threads (one scenario per call), timed like the other CPU
    legs; the GPU's moves, replicas and latency outcomes of those scenarios
    must equal the oracle's. With act_in, the oracle's replay under the same
    actuation model (delays in whole windows, rounded up)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle as O

    o = O.get()
    M = w.n_models
    cfg = w.trace_cfg()
    prof_all = O.pack_profiles(w.profile_columns())
    slo_all = O.pack_slo(w.slo_columns())
    svc_all = O.pack_svc(w.service_columns())
    sc_all = O.pack_scenarios(sc_cols)
    sample = list(range(min(n_sample, len(sc_all))))
    kw_t = lambda t: {}
    if act_in is not None:
        cfg = dict(cfg, budget=act_in["budget"])
        to_w = lambda ms: min(-(-ms // w.window_ms), w.n_windows + 1)
        kw_t = lambda t: {"wake_w": to_w(ACT_WAKE_MS), "sleep_w": to_w(ACT_SLEEP_MS), "footprint": act_in["g"][t],
                          "veto": act_in["veto"][t]}

    def one(s):
        c0 = time.thread_time()
        t = int(sc_all[s]["trace"])
        r = o.loop(cfg, prof_all[t * M:(t + 1) * M], sc_all[s:s + 1], slo_all[t * M:(t + 1) * M],
                   svc_all[t * M:(t + 1) * M], tables[t], move_cap=move_cap, **kw_t(t))
        return r, time.thread_time() - c0

    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=n_workers) as pool:
        results = list(pool.map(one, sample))
    wall = time.perf_counter() - t0
    cpu_s = sum(c for _, c in results)
    n_moves = out["n_moves"].cpu().numpy()
    r_final = out["r_final"].cpu().numpy()
    r_windows = out["r_windows"].cpu().numpy()
    moves = tre.unpack_moves(out["moves"]).reshape(-1, move_cap)
    st = stats.cpu().numpy().view(tre.LOOP_STATS_DTYPE).reshape(-1, M)
    bad = 0
    reqs = 0
    for s, (r, _) in zip(sample, results):
        reqs += len(tables[int(sc_all[s]["trace"])]["arrival_ms"])
        k = min(int(n_moves[s]), move_cap)
        ok = int(n_moves[s]) == r["n_moves"] and np.array_equal(r_final[s], r["r_final"]) and \
            np.array_equal(r_windows[s], r["r_windows"]) and \
            all(np.array_equal(moves[s][:k][f], r["moves"][:k][f]) for f in ("window", "path", "receiver", "donor")) and \
            all(np.array_equal(st[s][f], r["stats"][f]) for f in tre.LOOP_STATS_DTYPE.names)
        bad += 0 if ok else 1
    cpu = {"value": round(reqs / wall, 1), "unit": "requests/s", "cores": n_workers, **host_cpu(), "kind": "oracle",
           "sample": f"{len(sample)} of {len(sc_all)} scenarios ({reqs} requests): {wall:.1f} s wall on {n_workers} "
                     f"host threads (one scenario per oracle call), {cpu_s:.1f} s of their CPU time",
           "one_core_value": round(reqs / cpu_s, 1)}
    parity = {"scenarios_checked": len(sample), "mismatches": bad, "bit_exact": bad == 0}
    log(f"cpu oracle (closed loop): {cpu['value']:.3g} requests/s on {n_workers} threads; parity {parity}")
    return cpu, parity


def calibrate_main(args, w, dt, device, tre, torch, np):
    """One step = tre_eval_tss writing the per-cell smoothed TSS and flags,
    then tre_calibrate (request join, SLO attainment, theta fit) over the
    whole resident workload. Algorithmic bytes per launch: tss_stream 12 per
    event + 9 per cell written; calib_fill 0 (a few diagnostic words; the
    per-request records when asked for); calib_stream 16 per event
    (timestamp 8, request id 4, tokens 2, type 1, model 1) + 12 per cell
    (each counter zeroed, then read and written back once by its adds);
    calib_fallback 0 (the traces the stream could not finish, none on the
    standard workloads: its launches end at once); calib_fit 13 per cell
    (counter, TSS, flags)."""
    ev = device.load(dt, validate=True)
    prof = device.profiles(w)
    slo = device.slos(w)
    T, M, nW = ev.n_traces, ev.n_models, ev.n_windows
    cells = T * M * nW
    tss = {"tss64": torch.empty((T, nW, M), dtype=torch.float64, device="cuda"),
           "flags": torch.empty((T, nW, M), dtype=torch.uint8, device="cuda")}
    out = tre.calib_outputs(ev, dt.req_cap)
    log(f"calibration: {T} traces, {dt.n_events} events, {dt.n_arrive} requests ({dt.n_finish} finished), "
        f"req_cap {dt.req_cap}, workspace {out['ws'].numel() / 1e9:.1f} GB")

    def step():
        tre.tre_eval_tss(ev, prof, tss)
        tre.tre_calibrate(ev, slo, tss["tss64"], tss["flags"], out)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    tre.tre_set_timing(True)
    for k in CALIB_KERNELS:
        tre.tre_kernel_time(k)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    tre.tre_set_timing(False)
    step_ms = e0.elapsed_time(e1) / args.steps
    kms = {}
    for k in CALIB_KERNELS:
        tot, n = tre.tre_kernel_time(k)
        kms[k] = tot / max(n, 1)
    alg = {"tss_stream": ALG_BYTES_PER_EVENT * dt.n_events + 9 * cells,
           "calib_fill": 0,
           "calib_stream": 16 * dt.n_events + 12 * cells,
           "calib_fallback": 0,
           "calib_fit": 13 * cells}
    kernels = {k: {"ms": round(kms[k], 4), "alg_bytes": alg[k],
                   "gbs": round(alg[k] / (kms[k] / 1e3) / 1e9, 1) if kms[k] > 0 else None} for k in CALIB_KERNELS}
    kernels["calib_fallback"]["traces"] = dict(zip(("larger_table", "chunked"), tre.calib_fallback_traces(ev, out)))
    calib_only = [k for k in CALIB_KERNELS if k != "tss_stream"]
    dom = max(calib_only, key=lambda k: kms[k])
    roofline = {"bound": "hbm", "achieved": kernels[dom]["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(kernels[dom]["gbs"] / HBM_PEAK_GBS, 4),
                "traffic": calib_traffic_for(w.name, dt.n_events, dom), "kernel": dom,
                "kernel_ms": kernels[dom]["ms"], "alg_bytes_per_launch": alg[dom]}
    log("kernels " + ", ".join(f"{k} {kms[k]:.3f} ms" for k in CALIB_KERNELS) + f"; step {step_ms:.3f} ms")
    # the ordering check (outside the step): the fits again with the
    # concordant / discordant pair counts, from the step's counts
    tre.tre_set_timing(True)
    tre.tre_kernel_time("calib_order")
    tre.tre_calib_order(ev, slo, tss["tss64"], tss["flags"], out)
    o_ms, _ = tre.tre_kernel_time("calib_order")
    tre.tre_set_timing(False)
    fit_o = tre.unpack_fit(out["fit"])
    order = {"ms": round(o_ms, 4), "concordant": int(fit_o["concordant"].astype(np.int64).sum()),
             "discordant": int(fit_o["discordant"].astype(np.int64).sum())}
    log(f"ordering check: calib_order {o_ms:.3f} ms; concordant {order['concordant']}, "
        f"discordant {order['discordant']} pairs over all (trace, model)")
    cpu = parity = None
    if not args.no_cpu:
        n_s = max(1, int(np.searchsorted(np.cumsum(dt.counts), CPU_EVENT_BUDGET // 3, side="right")))
        cpu, parity = calib_cpu_leg(w, list(range(n_s)), out, tss, dt.req_cap, tre, args.threads)
    result = {
        "metric": "request-events/sec through TSS + calibration sweep (1 GPU)",
        "value": round(dt.n_events / (step_ms / 1e3), 1),
        "unit": "request-events/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic (seeded generator; the paper's traces are not available)",
        "config": {"workload": w.name, "traces": T, "models": M, "window_ms": w.window_ms,
                   "duration_s": w.duration_ms // 1000, "events": dt.n_events, "requests": dt.n_arrive,
                   "req_cap": dt.req_cap, "mode": "calibration"},
        "roofline": roofline, "kernels": kernels, "ordering_check": order, "cpu_baseline": cpu, "parity": parity,
    }
    print(json.dumps(result), flush=True)
    if args.copy_calib_gb > 0:
        del tss, out
        copy_calibration(args.copy_calib_gb, torch)
    ev.close()


STAGE_KERNELS = ("tss_stream", "stage_tss")


def stage_main(args, w, dt, device, tre, torch, np):
    """One step = tre_eval_stage over the whole resident workload: one pass
    over each trace's events writing the prefill and decode shares
    (binary64) and their flags, the tallies never leaving the chip.
    Algorithmic bytes per launch: 12 per event read + 17 per cell written.
    The two-pass path (tre_eval_tss writing the per-cell tallies, then
    tre_stage_tss) is timed beside it for comparison (24 bytes per cell
    written and read back) and must give the same shares in every cell."""
    ev = device.load(dt, validate=True)
    prof = device.profiles(w)
    T, M, nW = ev.n_traces, ev.n_models, ev.n_windows
    cells = T * M * nW
    out = tre.stage_outputs(ev, which=("stage64", "flags"))
    log(f"stage shares: {T} traces, {dt.n_events} events, {cells} cells")

    def timed(step, n, names):
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        tre.tre_set_timing(True)
        for k in names:
            tre.tre_kernel_time(k)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(n):
            step()
        e1.record(stream)
        torch.cuda.synchronize()
        tre.tre_set_timing(False)
        kms = {}
        for k in names:
            tot, c = tre.tre_kernel_time(k)
            kms[k] = tot / max(c, 1)
        return e0.elapsed_time(e1) / n, kms

    step_ms, kms = timed(lambda: tre.tre_eval_stage(ev, prof, out), args.steps, ("tss_stream",))
    k_ms = kms["tss_stream"]
    alg = ALG_BYTES_PER_EVENT * dt.n_events + 17 * cells
    log(f"one pass: step {step_ms:.3f} ms, tss_stream (stage) {k_ms:.3f} ms")
    # the two-pass path, for comparison
    tal = tre.tss_outputs(ev, which=("prefill", "decode", "a_int", "w_int"))
    two = tre.stage_outputs(ev, which=("stage64", "flags"))
    two_ms, two_k = timed(lambda: (tre.tre_eval_tss(ev, prof, tal), tre.tre_stage_tss(ev, prof, tal, two)),
                          min(args.steps, 3), STAGE_KERNELS)
    same = bool(torch.equal(two["stage64"].view(torch.int64), out["stage64"].view(torch.int64)) and
                torch.equal(two["flags"], out["flags"]))
    log(f"two pass: step {two_ms:.3f} ms ({', '.join(f'{k} {v:.3f} ms' for k, v in two_k.items())}); "
        f"same shares: {same}")
    del tal, two
    torch.cuda.empty_cache()
    two_alg = {"tss_stream": ALG_BYTES_PER_EVENT * dt.n_events + 24 * cells, "stage_tss": 41 * cells}
    two_pass = {"ms_per_step": round(two_ms, 4), "same_shares": same,
                "kernels": {k: {"ms": round(two_k[k], 4), "alg_bytes": two_alg[k],
                                "gbs": round(two_alg[k] / (two_k[k] / 1e3) / 1e9, 1) if two_k[k] > 0 else None}
                            for k in STAGE_KERNELS}}
    gbs = alg / (k_ms / 1e3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": stage_traffic_for(w.name, cells),
                "kernel": "tss_stream (stage)", "kernel_ms": round(k_ms, 4), "alg_bytes_per_launch": alg}
    cpu = parity = None
    if not args.no_cpu:
        n_s = max(1, int(np.searchsorted(np.cumsum(dt.counts), CPU_EVENT_BUDGET // 3, side="right")))
        cpu, parity = stage_cpu_leg(w, list(range(n_s)), out, args.threads)
    result = {
        "metric": "request-events/sec through stage-aware shares (1 GPU)",
        "value": round(dt.n_events / (step_ms / 1e3), 1),
        "unit": "request-events/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic (seeded generator; the paper's traces are not available)",
        "config": {"workload": w.name, "traces": T, "models": M, "window_ms": w.window_ms,
                   "duration_s": w.duration_ms // 1000, "events": dt.n_events, "cells": cells, "mode": "stage"},
        "roofline": roofline, "two_pass": two_pass, "cpu_baseline": cpu, "parity": parity,
    }
    print(json.dumps(result), flush=True)
    if args.copy_calib_gb > 0:
        del out
        torch.cuda.empty_cache()
        copy_calibration(args.copy_calib_gb, torch)
    ev.close()


def stage_traffic_for(workload_name: str, cells: int):
    """HBM bytes per one-pass stage launch (tss_stream's stage
    instantiation) from committed counters taken on this kernel source and
    workload; else None."""
    try:
        t = json.load(open(os.path.join(ROOT, "profiles", "stage_traffic.json")))
    except (OSError, ValueError):
        return None
    if t.get("kernel_sha") != kernel_sha() or t.get("workload") != workload_name or t.get("cells") != cells:
        return None
    return t.get("traffic_bytes_per_launch", {}).get("tss_stream_stage")


def stage_cpu_leg(w, sample, out, threads):
    """The oracle's tallies and stage shares of the sample traces on a pool
    of host threads; the GPU's shares (bit for bit) and flags of those
    traces must equal the oracle's."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle as O

    o = O.get()
    M = w.n_models
    prof_all = O.pack_profiles(w.profile_columns(max(sample) + 1))
    n_workers = max(1, min(CPU_WORKERS, os.cpu_count() or 1))

    def one(ev, t):
        c0 = time.thread_time()
        p = prof_all[t * M:(t + 1) * M]
        r = o.stage_tss(o.tss_trace(ev, w.window_ms, w.duration_ms, p), w.window_ms, p)
        return r, time.thread_time() - c0

    wall = cpu_s = 0.0
    events = 0
    bad = 0
    batch = 4 * n_workers
    with ThreadPoolExecutor(max_workers=n_workers) as pool:
        for b0 in range(0, len(sample), batch):
            tr = sample[b0:b0 + batch]
            host = w.generate(tr[0], tr[-1] + 1, threads=threads)
            evs = [host.trace(i) for i in range(len(tr))]
            t0 = time.perf_counter()
            results = list(pool.map(one, evs, tr))
            wall += time.perf_counter() - t0
            for ev, t, (rf, c) in zip(evs, tr, results):
                cpu_s += c
                events += len(ev["ts"])
                g64 = out["stage64"][t].cpu().numpy()
                gfl = out["flags"][t].cpu().numpy()
                ok = np.array_equal(g64.view(np.uint64), rf["S"].view(np.uint64)) and np.array_equal(gfl, rf["flags"])
                bad += 0 if ok else 1
            del host, evs
    cpu = {"value": round(events / wall, 1), "unit": "request-events/s", "cores": n_workers, **host_cpu(), "kind": "oracle",
           "sample": f"{len(sample)} of {w.n_traces} traces ({events} events): {wall:.1f} s wall on {n_workers} "
                     f"host threads (one trace per oracle call: tallies, TSS and stage shares), {cpu_s:.1f} s of "
                     f"their CPU time",
           "one_core_value": round(events / cpu_s, 1)}
    parity = {"traces_checked": len(sample), "mismatches": bad, "bit_exact": bad == 0}
    log(f"cpu oracle (stage shares): {cpu['value']:.3g} events/s on {n_workers} threads; parity {parity}")
    return cpu, parity


def calib_traffic_for(workload_name: str, events: int, kernel: str):
    """HBM bytes per launch of a calibration kernel from committed counters
    taken on this kernel source and workload; else None."""
    try:
        t = json.load(open(os.path.join(ROOT, "profiles", "calib_traffic.json")))
    except (OSError, ValueError):
        return None
    src = os.path.join(ROOT, "paper_2609_29160_amd", "csrc", "calib.hip")
    if t.get("kernel_sha") != kernel_sha(src) or t.get("workload") != workload_name or t.get("events") != events:
        return None
    if kernel == "tss_stream" and t.get("tre_sha") != kernel_sha():  # tss_stream's own source
        return None
    return t.get("traffic_bytes_per_launch", {}).get(kernel)


def flat_read_rate(col, torch, reps=3):
    """What a plain contiguous read of a resident column reaches on this
    GPU (torch's sum over the int64 ts column, after the timed region): the
    ceiling beside the kernel's roofline fraction, not part of `value`."""
    col.sum()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        col.sum()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = col.numel() * col.element_size()
    return {"what": "torch.sum over the resident ts column (a flat read)", "bytes": nbytes, "ms": round(ms, 3),
            "gbs": round(nbytes / (ms / 1e3) / 1e9, 1)}


def copy_calibration(gb, torch):
    """A plain device copy of known size, for scaling the traffic counters."""
    n = int(gb * 1e9) // 4
    src = torch.ones(n, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy calibration: 3 x {4 * n} bytes read + written")


def calib_cpu_leg(w, sample, out, tss, req_cap, tre, threads):
    """The oracle's calibration (TSS, join, attainment, fit) of the sample
    traces on a pool of host threads, timed like the replay's CPU leg; the
    GPU's counts and fits of those traces must equal the oracle's."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle as O

    o = O.get()
    M = w.n_models
    prof_all = O.pack_profiles(w.profile_columns(max(sample) + 1))
    slo_all = O.pack_slo(w.slo_columns(max(sample) + 1))
    n_workers = max(1, min(CPU_WORKERS, os.cpu_count() or 1))

    def one(ev, t):
        c0 = time.thread_time()
        r = o.calibrate(ev, w.window_ms, w.duration_ms, prof_all[t * M:(t + 1) * M], slo_all[t * M:(t + 1) * M],
                        req_cap)
        return {"judged": r["judged"], "ok": r["ok"], "fit": r["fit"]}, time.thread_time() - c0

    wall = cpu_s = 0.0
    events = 0
    refs = {}
    batch = 4 * n_workers
    with ThreadPoolExecutor(max_workers=n_workers) as pool:
        for b0 in range(0, len(sample), batch):
            tr = sample[b0:b0 + batch]
            host = w.generate(tr[0], tr[-1] + 1, threads=threads)
            evs = [host.trace(i) for i in range(len(tr))]
            t0 = time.perf_counter()
            results = list(pool.map(one, evs, tr))
            wall += time.perf_counter() - t0
            for ev, t, (rf, c) in zip(evs, tr, results):
                refs[t] = rf
                cpu_s += c
                events += len(ev["ts"])
            del host, evs
    fit = tre.unpack_fit(out["fit"]).reshape(-1, M)
    bad = 0
    for t, rf in refs.items():
        cnt = out["counts"][t].cpu().numpy().view(np.uint32)
        ok = np.array_equal(cnt >> 16, rf["judged"]) and np.array_equal(cnt & 0xFFFF, rf["ok"])
        ok = ok and np.array_equal(fit[t]["theta"].view(np.uint64), rf["fit"]["theta"].view(np.uint64))
        for k in ("n_cand", "n_healthy", "n_above", "healthy_above", "concordant", "discordant"):
            ok = ok and np.array_equal(fit[t][k], rf["fit"][k])
        bad += 0 if ok else 1
    cpu = {"value": round(events / wall, 1), "unit": "request-events/s", "cores": n_workers, **host_cpu(), "kind": "oracle",
           "sample": f"{len(sample)} of {w.n_traces} traces ({events} events): {wall:.1f} s wall on {n_workers} "
                     f"host threads (one trace per oracle call), {cpu_s:.1f} s of their CPU time",
           "one_core_value": round(events / cpu_s, 1)}
    parity = {"traces_checked": len(refs), "mismatches": bad, "bit_exact": bad == 0}
    log(f"cpu oracle (calibration): {cpu['value']:.3g} events/s on {n_workers} threads; parity {parity}")
    return cpu, parity


def actuation_inputs(w):
    """Footprints (1 or 2 GPUs per replica, [trace][model]) and the GPU
    budget that holds every trace's initial replicas with 8 GPUs to spare."""
    import numpy as np

    rng = np.random.default_rng(ACT_SEED)
    g = rng.integers(1, 3, (w.n_traces, w.n_models)).astype(np.int32)
    r_init = np.asarray(w.profile_columns()["r_init"]).reshape(w.n_traces, w.n_models)
    return {"g": g, "budget": int((g * r_init).sum(axis=1).max()) + 8}


CLASS_GPUS = {"7B": 1, "13B": 1, "34B": 2, "70B": 4}  # GPUs per replica of each model class


def replica_bound(g, budget, r_cap):
    """The most replicas a model set can hold at once: each model below
    r_cap + 1 replicas, their footprints within the GPU budget; filling the
    budget from the smallest footprint up reaches it."""
    n, left = 0, budget
    for gm in sorted(int(x) for x in g):
        k = min(r_cap, left // gm)
        n += k
        left -= k * gm
    return n


def loop_actuation_inputs(w, r_cap=16):
    """The closed loop's actuation model: footprints by model class
    ([trace][model]), the GPU budget that holds every trace's initial
    replicas with 8 GPUs to spare, and the most replicas the budget and the
    replica cap allow at once, declared to tre_loop_act (it sizes the slot
    pool)."""
    import numpy as np

    g1 = np.array([CLASS_GPUS[c] for c in w.model_classes], np.int32)
    g = np.ascontiguousarray(np.broadcast_to(g1, (w.n_traces, w.n_models)))
    r_init = np.asarray(w.profile_columns()["r_init"]).reshape(w.n_traces, w.n_models)
    budget = int((g * r_init).sum(axis=1).max()) + 8
    bound = max(replica_bound(row, budget, r_cap) for row in {tuple(r) for r in g})
    return {"g": g, "budget": budget, "max_replicas": bound}


def actuation_vetoes(w, n_ticks):
    """Donor-release veto masks [trace][tick]: on 10% of the ticks, a random
    subset of the models."""
    import numpy as np

    rng = np.random.default_rng(ACT_SEED + 1)
    full = np.uint64((1 << w.n_models) - 1) if w.n_models < 64 else np.uint64(0xFFFFFFFFFFFFFFFF)
    veto = rng.integers(0, 1 << 63, (w.n_traces, n_ticks), dtype=np.int64).astype(np.uint64) & full
    veto[rng.random(veto.shape) >= 0.1] = 0
    return veto


def cpu_leg(w, sample, sc_cols, out, move_cap, tre, threads, act_in=None):
    """Time the oracle on the sample traces and compare the GPU's decisions
    for the scenarios on those traces.  The sample's host columns are
    generated again in batches (same seeds as the device copy); the oracle
    calls of a batch run on a pool of host threads (one trace per call, the
    oracle itself is single-threaded), and only those calls are timed: wall
    time of the pool for the all-core rate, the calls' own thread CPU time
    for the one-core rate."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle as O

    o = O.get()
    M = w.n_models
    prof_all = O.pack_profiles(w.profile_columns(max(sample) + 1))
    sc_all = O.pack_scenarios(sc_cols)
    cfg = w.trace_cfg()
    by_trace = {}
    for s, t in enumerate(sc_cols["trace"]):
        by_trace.setdefault(int(t), []).append(s)
    n_workers = max(1, min(CPU_WORKERS, os.cpu_count() or 1))

    if act_in is not None:
        cfg = dict(cfg, budget=act_in["budget"])
        # delays in whole windows: rounded up, at most one past the end
        n_w = w.duration_ms // w.window_ms
        wake_w, sleep_w = (min(-(-ms // w.window_ms), n_w + 1) for ms in (ACT_WAKE_MS, ACT_SLEEP_MS))

    def one(ev, t):
        c0 = time.thread_time()
        prof = prof_all[t * M:(t + 1) * M]
        r = o.tss_trace(ev, w.window_ms, w.duration_ms, prof)
        if act_in is None:
            refs = {s: o.control(cfg, prof, r["S"], r["flags"], sc_all[s:s + 1], move_cap)
                    for s in by_trace.get(t, [])}
        else:
            refs = {s: o.control_act(cfg, prof, r["S"], r["flags"], sc_all[s:s + 1], wake_w, sleep_w,
                                     footprint=act_in["g"][t], veto=act_in["veto"][t], move_cap=move_cap)
                    for s in by_trace.get(t, [])}
        return refs, time.thread_time() - c0

    wall = 0.0
    cpu_s = 0.0
    logical = 0
    events = 0
    refs = {}
    batch = 4 * n_workers
    with ThreadPoolExecutor(max_workers=n_workers) as pool:
        for b0 in range(0, len(sample), batch):
            tr = sample[b0:b0 + batch]
            host = w.generate(tr[0], tr[-1] + 1, threads=threads)
            evs = [host.trace(i) for i in range(len(tr))]
            t0 = time.perf_counter()
            results = list(pool.map(one, evs, tr))
            wall += time.perf_counter() - t0
            for ev, t, (rf, c) in zip(evs, tr, results):
                refs.update(rf)
                cpu_s += c
                events += len(ev["ts"])
                logical += len(ev["ts"]) * len(by_trace.get(t, []))
            del host, evs
    # parity of the last timed sweep on the sampled scenarios
    n_moves = out["n_moves"].cpu().numpy()
    r_final = out["r_final"].cpu().numpy()
    r_windows = out["r_windows"].cpu().numpy()
    moves = tre.unpack_moves(out["moves"]).reshape(-1)
    bad = 0
    for s, ref in refs.items():
        k = int(n_moves[s])
        ok = k == ref["n_moves"] and np.array_equal(r_final[s], ref["r_final"]) and \
            np.array_equal(r_windows[s], ref["r_windows"])
        if ok:
            got = moves[s * move_cap:s * move_cap + min(k, move_cap)]
            exp = ref["moves"][:min(k, move_cap)]
            ok = all(np.array_equal(got[f], exp[f]) for f in ("window", "path", "receiver", "donor"))
        bad += 0 if ok else 1
    cpu = {"value": round(logical / wall, 1), "unit": "request-events/s", "cores": n_workers, **host_cpu(), "kind": "oracle",
           "sample": f"{len(sample)} of {w.n_traces} traces ({events} events), {len(refs)} scenarios: "
                     f"{wall:.1f} s wall on {n_workers} host threads (one trace per oracle call), "
                     f"{cpu_s:.1f} s of their CPU time",
           "one_core_value": round(logical / cpu_s, 1)}
    parity = {"scenarios_checked": len(refs), "mismatches": bad, "bit_exact": bad == 0}
    log(f"cpu oracle: {cpu['value']:.3g} events/s on {n_workers} threads "
        f"({cpu['one_core_value']:.3g} on one); parity {parity}")
    return cpu, parity


if __name__ == "__main__":
    main()
