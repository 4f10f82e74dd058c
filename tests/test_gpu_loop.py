"""GPU parity of the closed-loop replay (tre_loop) against the oracle's.

For every scenario: the move log, final replicas, replica-window sums, the
per-model latency outcomes (arrived, started, judged, SLO met, E2E sum and
maximum) and the per-window smoothed TSS (bit for bit) must equal the
oracle's, and no event may fall outside the ring of future windows.

Inputs: the tiny and bursty workloads' request tables (the same arrivals and
lengths as their traces) under scenario tables with 0 to 4 moves per tick,
spare budget and replica caps that bind; budgets above n_models * r_cap; an
empty request table and models without requests; the oracle's hand cases;
1, 17 and 64 models; one and three slots per replica; argument errors
(including slot heaps beyond the LDS and negative actuation delays).

tre_loop_act against the oracle's closed loop under the actuation model, to
the same bar: zero delays with unit footprints and no vetoes equal to
tre_loop; the paper's wake and sleep times (1.31 s, 1.87 s) with footprints
of 1 or 2 GPUs and vetoes on 20% of the ticks, with and without idle GPUs;
delays longer than the trace; 1, 17 and 64 models; the oracle's hand case.
"""
import sys

import numpy as np
import pytest

import oracle as O
import tracegen as tg

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


def _rows(cols, t, M, dtype):
    a = np.zeros(M, dtype)
    for k in dtype.names:
        a[k] = cols[k][t * M:(t + 1) * M]
    return a


def _n_ticks(cfg):
    nW = cfg["duration_ms"] // cfg["window_ms"]
    return sum(1 for w in range(nW) if ((w + 1) * cfg["window_ms"]) % cfg["fast_period_ms"] == 0
               or ((w + 1) * cfg["window_ms"]) % cfg["slow_period_ms"] == 0)


def _check(lib, name, cfg, tables, prof_cols, slo_cols, svc_cols, sc_cols, spr=8, r_cap=16, act=None,
           max_replicas=0):
    """act: (wake_ms, sleep_ms, footprint [T][M] int32 or None, veto [T][n_ticks] uint64 or None) runs
    tre_loop_act against the oracle's closed loop with the actuation model."""
    tre, device, torch = lib
    M = cfg["n_models"]
    T = len(tables)
    nW = cfg["duration_ms"] // cfg["window_ms"]
    svc = np.zeros(T * M, tre.SERVICE_DTYPE)
    for k in tre.SERVICE_DTYPE.names:
        svc[k] = svc_cols[k]
    slo = np.zeros(T * M, tre.SLO_DTYPE)
    for k in tre.SLO_DTYPE.names:
        slo[k] = slo_cols[k]
    rq, keep = tre.loop_requests(tables, M, svc, slo, slots_per_replica=spr, r_cap=r_cap, max_replicas=max_replicas)
    prof = tre.pack(prof_cols, tre.PROFILE_DTYPE)
    sc = tre.pack(sc_cols, tre.SCENARIO_DTYPE)
    n_sc = len(sc_cols["trace"])
    move_cap = max(1, _n_ticks(cfg) * int(np.max(sc_cols["max_moves"])))
    out = tre.ctl_outputs(_Ev(T, M, nW), n_sc, move_cap)
    stats = torch.zeros(n_sc * M * tre.LOOP_STATS_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    tss = torch.zeros((n_sc, nW, M), dtype=torch.float64, device="cuda")
    ws = torch.empty(tre.tre_loop_workspace_size(cfg, rq, n_sc), dtype=torch.uint8, device="cuda")
    if act is None:
        tre.tre_loop(cfg, T, rq, prof, sc, out, stats, ws, tss64=tss)
    else:
        wake_ms, sleep_ms, fp, veto = act
        fp_t = None if fp is None else torch.from_numpy(np.ascontiguousarray(fp, np.int32)).cuda()
        v_t = None if veto is None else torch.from_numpy(np.ascontiguousarray(veto, np.uint64).view(np.int64)).cuda()
        tre.tre_loop_act(cfg, T, rq, prof, sc, tre.actuation(wake_ms, sleep_ms, fp_t, v_t), out, stats, ws, tss64=tss)
        cap = nW + 1
        to_w = lambda ms: cap if ms > cap * cfg["window_ms"] else -(-ms // cfg["window_ms"])
    torch.cuda.synchronize()
    assert int(ws[:8].cpu().numpy().view(np.uint64)[0]) == 0, f"{name}: events beyond the ring"
    moves = tre.unpack_moves(out["moves"]).reshape(n_sc, move_cap)
    st = stats.cpu().numpy().view(tre.LOOP_STATS_DTYPE).reshape(n_sc, M)
    S = tss.cpu().numpy()
    o = O.get()
    total_moves = 0
    for s in range(n_sc):
        t = int(sc_cols["trace"][s])
        row = np.zeros(1, O.SCENARIO_DTYPE)
        for k in O.SCENARIO_DTYPE.names:
            row[k] = sc_cols[k][s]
        kw = {}
        if act is not None:
            kw = {"wake_w": to_w(wake_ms), "sleep_w": to_w(sleep_ms),
                  "footprint": np.ones(M, np.int32) if fp is None else np.asarray(fp)[t],
                  "veto": None if veto is None else np.asarray(veto, np.uint64)[t]}
        ref = o.loop(cfg, _rows(prof_cols, t, M, O.PROFILE_DTYPE), row, _rows(slo_cols, t, M, O.SLO_DTYPE),
                     _rows(svc_cols, t, M, O.SVC_DTYPE), tables[t], spr=spr, r_cap=r_cap, move_cap=move_cap,
                     want_tss=True, **kw)
        what = f"{name} scenario {s}"
        n = int(out["n_moves"][s])
        assert n == ref["n_moves"], f"{what}: {n} moves vs {ref['n_moves']}"
        k = min(n, move_cap)
        for f in ("window", "path", "receiver", "donor"):
            assert np.array_equal(moves[s][:k][f], ref["moves"][:k][f]), f"{what}: moves ({f})"
        assert np.array_equal(out["r_final"][s].cpu().numpy(), ref["r_final"]), f"{what}: r_final"
        assert np.array_equal(out["r_windows"][s].cpu().numpy(), ref["r_windows"]), f"{what}: r_windows"
        for f in tre.LOOP_STATS_DTYPE.names:
            assert np.array_equal(st[s][f], ref["stats"][f]), f"{what}: stats {f} {st[s][f]} vs {ref['stats'][f]}"
        assert np.array_equal(S[s].view(np.uint64), ref["S"].view(np.uint64)), f"{what}: TSS"
        total_moves += n
    return total_moves


class _Ev:
    """The shape ctl_outputs needs (models), without an events handle."""

    def __init__(self, T, M, nW):
        self.n_traces, self.n_models, self.n_windows = T, M, nW


def _scenarios(rng, n, n_traces, ks=(0, 1, 2, 4)):
    return {"trace": (np.arange(n) % n_traces).astype(np.uint32),
            "max_moves": np.array([ks[i % len(ks)] for i in range(n)], np.uint32),
            "theta_scale": rng.uniform(0.5, 2.0, n),
            "tau_crit_override": np.where(rng.random(n) < 0.5, -1.0, rng.uniform(0.2, 0.8, n))}


def test_tiny(lib):
    w = tg.standard(0)
    tables = [w.requests(0)]
    rng = np.random.default_rng(1)
    cfg = dict(w.trace_cfg(), budget=w.budget + 2)
    n = _check(lib, "tiny", cfg, tables, w.profile_columns(1), w.slo_columns(1), w.service_columns(1),
               _scenarios(rng, 8, 1))
    assert n > 0


def test_bursty_spare_budget_and_binding_cap(lib):
    w = tg.standard(1).scaled(duration_ms=900_000)
    tables = [w.requests(0)]
    rng = np.random.default_rng(2)
    for extra, r_cap in ((0, 16), (3, 16), (3, 5)):
        cfg = dict(w.trace_cfg(), budget=w.budget + extra)
        say(f"bursty budget +{extra}, r_cap {r_cap}")
        n = _check(lib, f"bursty-{extra}-{r_cap}", cfg, tables, w.profile_columns(1), w.slo_columns(1),
                   w.service_columns(1), _scenarios(rng, 12, 1), r_cap=r_cap)
        assert n > 0


def test_several_traces(lib):
    w = tg.standard(3).scaled(n_traces=3, duration_ms=600_000)
    tables = [w.requests(t) for t in range(3)]
    rng = np.random.default_rng(3)
    cfg = dict(w.trace_cfg(), budget=w.budget + 4)
    _check(lib, "diverse-3tr", cfg, tables, w.profile_columns(3), w.slo_columns(3), w.service_columns(3),
           _scenarios(rng, 9, 3))


def test_wide_service_bounds(lib):
    """A model whose prompt tokens take 2.2 s each: a full prompt chunk's
    tokens * us then passes 2^32, so the remainder-chunk times take their
    64-bit path for every model; results as the oracle's."""
    w = tg.standard(0)
    tables = [w.requests(0)]
    rng = np.random.default_rng(14)
    svc = {k: np.array(v, copy=True) for k, v in w.service_columns(1).items()}
    svc["prefill_us"][0] = 2_200_000
    svc["decode_us"][-1] = svc["decode_us"][-1] * 50
    assert 2048 * int(svc["prefill_us"].max()) + 999 >= 1 << 32
    cfg = dict(w.trace_cfg(), budget=w.budget + 2)
    _check(lib, "wide-service", cfg, tables, w.profile_columns(1), w.slo_columns(1), svc, _scenarios(rng, 8, 1))


def test_slots_per_replica(lib):
    w = tg.standard(0)
    tables = [w.requests(0)]
    rng = np.random.default_rng(4)
    for spr in (1, 3):
        cfg = dict(w.trace_cfg(), budget=w.budget + 1)
        _check(lib, f"spr{spr}", cfg, tables, w.profile_columns(1), w.slo_columns(1), w.service_columns(1),
               _scenarios(rng, 4, 1), spr=spr)


def test_hand_cases(lib):
    """The oracle's hand-derived cases, through the GPU."""
    for r_cap in (3, 2):
        cfg = {"window_ms": 100, "duration_ms": 1000, "fast_period_ms": 100, "slow_period_ms": 100,
               "n_models": 2, "budget": 3}
        prof = {"w_p": np.full(2, 0.5), "w_q": np.full(2, 2.0), "alpha": np.ones(2), "theta": np.full(2, 1e12),
                "tau_crit": np.full(2, 0.5), "tau_surplus": np.full(2, 1.5), "r_min": np.zeros(2, np.int32),
                "r_init": np.ones(2, np.int32)}
        slo = {"ttft_ms": np.full(2, 1e9), "tpot_ms": np.full(2, 1e9), "e2e_ms": np.full(2, 1e9),
               "attain_q": np.full(2, 0.95), "reliability": np.full(2, 0.9)}
        svc = {"prefill_us": np.full(2, 1000, np.uint32), "decode_us": np.full(2, 10000, np.uint32)}
        table = {"arrival_ms": np.zeros(3, np.int64), "model": np.zeros(3, np.uint8), "prompt": np.ones(3, np.uint16),
                 "output": np.full(3, 24, np.uint16)}
        sc = {"trace": np.zeros(1, np.uint32), "max_moves": np.ones(1, np.uint32), "theta_scale": np.ones(1),
              "tau_crit_override": -np.ones(1)}
        n = _check(lib, f"hand-cap{r_cap}", cfg, [table], prof, slo, svc, sc, spr=1, r_cap=r_cap)
        assert n == (2 if r_cap == 3 else 1)


def test_model_counts(lib):
    for M in (1, 17, 64):
        w = tg.Workload(name=f"m{M}", n_traces=1, model_classes=[["7B", "13B", "34B", "70B"][m % 4] for m in range(M)],
                        interactive=[m % 2 == 0 for m in range(M)], r_init=[2] * M, budget=2 * M + 3,
                        window_ms=500, duration_ms=600_000, process="mmpp2", rate=[0.8] * M,
                        proc_params={"mmpp_mult": 6.0, "mmpp_dwell_s": 60.0}, seed=60 + M)
        tables = [w.requests(0)]
        rng = np.random.default_rng(M)
        say(f"M {M}: {len(tables[0]['arrival_ms'])} requests")
        _check(lib, f"M{M}", w.trace_cfg(), tables, w.profile_columns(1), w.slo_columns(1), w.service_columns(1),
               _scenarios(rng, 4, 1))


def test_budget_above_the_replica_caps(lib):
    """A budget larger than n_models * r_cap: the heaps' pool holds
    n_models * r_cap replicas and the idle budget never runs out."""
    w = tg.standard(0)
    tables = [w.requests(0)]
    rng = np.random.default_rng(7)
    for r_cap, spr in ((2, 8), (4, 1), (3, 3)):
        cfg = dict(w.trace_cfg(), budget=3 * r_cap + 5)
        prof = dict(w.profile_columns(1))
        prof["r_init"] = np.minimum(np.asarray(prof["r_init"]), r_cap).astype(np.int32)
        say(f"r_cap {r_cap}, slots per replica {spr}, budget {cfg['budget']}")
        _check(lib, f"cap{r_cap}-spr{spr}", cfg, tables, prof, w.slo_columns(1), w.service_columns(1),
               _scenarios(rng, 6, 1, ks=(1, 2, 4)), spr=spr, r_cap=r_cap)


def test_empty_tables(lib):
    """A trace with no requests, and models with none in the others."""
    w = tg.standard(3).scaled(n_traces=3, duration_ms=300_000)
    tables = [w.requests(t) for t in range(3)]
    empty = {k: v[:0] for k, v in tables[0].items()}
    keep = np.asarray(tables[2]["model"]) % 4 != 1  # models 1, 5, 9, 13 get nothing
    thin = {k: np.asarray(v)[keep] for k, v in tables[2].items()}
    tables = [tables[1], empty, thin]
    rng = np.random.default_rng(9)
    cfg = dict(w.trace_cfg(), budget=w.budget + 2)
    _check(lib, "empty", cfg, tables, w.profile_columns(3), w.slo_columns(3), w.service_columns(3),
           _scenarios(rng, 9, 3))


def _act_model(rng, n_traces, M, n_ticks, veto_frac=0.2):
    fp = rng.integers(1, 3, (n_traces, M)).astype(np.int32)
    veto = np.frombuffer(rng.bytes(8 * n_traces * n_ticks), np.uint64).reshape(n_traces, n_ticks).copy()
    veto &= np.uint64((1 << M) - 1)
    veto[rng.random(veto.shape) > veto_frac] = 0
    return fp, veto


def test_actuation_zero_delays_equal_the_plain_loop(lib):
    w = tg.standard(0)
    tables = [w.requests(0)]
    rng = np.random.default_rng(41)
    cfg = dict(w.trace_cfg(), budget=w.budget + 2)
    sc = _scenarios(rng, 8, 1)
    a = _check(lib, "act0", cfg, tables, w.profile_columns(1), w.slo_columns(1), w.service_columns(1), sc,
               act=(0, 0, np.ones((1, w.n_models), np.int32), np.zeros((1, _n_ticks(cfg)), np.uint64)))
    b = _check(lib, "plain", cfg, tables, w.profile_columns(1), w.slo_columns(1), w.service_columns(1), sc)
    assert a == b > 0


def test_actuation_paper_delays(lib):
    """The paper's wake and sleep times (1.31 s, 1.87 s: 3 and 4 windows of
    500 ms), footprints of 1 or 2 GPUs, vetoes on 20% of the ticks."""
    w = tg.standard(1).scaled(duration_ms=900_000)
    tables = [w.requests(0)]
    rng = np.random.default_rng(42)
    cfg = dict(w.trace_cfg())
    fp, veto = _act_model(rng, 1, w.n_models, _n_ticks(cfg))
    r_init = np.asarray(w.profile_columns(1)["r_init"])
    for extra in (0, 6):
        cfg["budget"] = int((fp[0] * r_init).sum()) + extra
        say(f"paper delays, budget {cfg['budget']} GPUs")
        n = _check(lib, f"act-paper-{extra}", cfg, tables, w.profile_columns(1), w.slo_columns(1),
                   w.service_columns(1), _scenarios(rng, 12, 1), r_cap=10, act=(1310, 1870, fp, veto))
        assert n > 0


def test_actuation_delays_past_the_trace_and_model_counts(lib):
    w = tg.standard(0)
    tables = [w.requests(0)]
    rng = np.random.default_rng(43)
    cfg = dict(w.trace_cfg(), budget=w.budget + 3)
    _check(lib, "act-long", cfg, tables, w.profile_columns(1), w.slo_columns(1), w.service_columns(1),
           _scenarios(rng, 4, 1), act=(10 ** 9, 5000, None, None))
    for M in (1, 17, 64):
        wm = tg.Workload(name=f"m{M}", n_traces=1, model_classes=[["7B", "13B", "34B", "70B"][m % 4] for m in range(M)],
                         interactive=[m % 2 == 0 for m in range(M)], r_init=[2] * M, budget=2 * M + 3,
                         window_ms=500, duration_ms=600_000, process="mmpp2", rate=[0.8] * M,
                         proc_params={"mmpp_mult": 6.0, "mmpp_dwell_s": 60.0}, seed=70 + M)
        tables = [wm.requests(0)]
        c = wm.trace_cfg()
        fp, veto = _act_model(rng, 1, M, _n_ticks(c))
        c["budget"] = int((fp[0] * 2).sum()) + 3
        say(f"actuation, M {M}")
        _check(lib, f"act-M{M}", c, tables, wm.profile_columns(1), wm.slo_columns(1), wm.service_columns(1),
               _scenarios(rng, 4, 1), act=(1000, 1500, fp, veto))


def test_actuation_hand_case(lib):
    """The oracle's hand case: wake 2 windows, sleep 1 window."""
    cfg = {"window_ms": 100, "duration_ms": 1000, "fast_period_ms": 100, "slow_period_ms": 100,
           "n_models": 2, "budget": 3}
    prof = {"w_p": np.full(2, 0.5), "w_q": np.full(2, 2.0), "alpha": np.ones(2), "theta": np.full(2, 1e12),
            "tau_crit": np.full(2, 0.5), "tau_surplus": np.full(2, 1.5), "r_min": np.zeros(2, np.int32),
            "r_init": np.ones(2, np.int32)}
    slo = {"ttft_ms": np.full(2, 1e9), "tpot_ms": np.full(2, 1e9), "e2e_ms": np.full(2, 1e9),
           "attain_q": np.full(2, 0.95), "reliability": np.full(2, 0.9)}
    svc = {"prefill_us": np.full(2, 1000, np.uint32), "decode_us": np.full(2, 10000, np.uint32)}
    table = {"arrival_ms": np.zeros(3, np.int64), "model": np.zeros(3, np.uint8), "prompt": np.ones(3, np.uint16),
             "output": np.full(3, 24, np.uint16)}
    sc = {"trace": np.zeros(1, np.uint32), "max_moves": np.ones(1, np.uint32), "theta_scale": np.ones(1),
          "tau_crit_override": -np.ones(1)}
    n = _check(lib, "act-hand", cfg, [table], prof, slo, svc, sc, spr=1, r_cap=3, act=(200, 100, None, None))
    assert n == 2


CLASS_GPUS = {"7B": 1, "13B": 1, "34B": 2, "70B": 4}


def test_declared_replica_bound(lib):
    """Footprints by model class and a declared bound on the replicas
    holding slots (the most the GPU budget and the replica cap allow): the
    same results as the oracle's; and bounds that a replay exceeds are
    counted, never written past the pool."""
    tre, device, torch = lib
    w = tg.standard(1).scaled(duration_ms=900_000)
    tables = [w.requests(0)]
    rng = np.random.default_rng(44)
    M = w.n_models
    fp = np.array([[CLASS_GPUS[c] for c in w.model_classes]], np.int32)
    r_init = np.asarray(w.profile_columns(1)["r_init"])
    spare = 6
    cfg = dict(w.trace_cfg(), budget=int((fp[0] * r_init).sum()) + spare)
    # the most replicas the budget allows with at most r_cap per model:
    # filled from the smallest footprint up (a donor's excess GPUs can wake
    # further small replicas, so the initial count plus the idle GPUs is no
    # bound)
    bound, left = 0, cfg["budget"]
    for gm in sorted(fp[0].tolist()):
        k = min(10, left // gm)
        bound, left = bound + k, left - k * gm
    assert bound < cfg["budget"]
    sc_cols = _scenarios(rng, 12, 1)
    act = (1310, 1870, fp, None)
    n = _check(lib, "bound", cfg, tables, w.profile_columns(1), w.slo_columns(1), w.service_columns(1), sc_cols,
               r_cap=10, act=act, max_replicas=bound)
    assert n > 0
    # too small: the initial replicas cut, or the pool's wakes beyond it
    svc = np.zeros(M, tre.SERVICE_DTYPE)
    for k in tre.SERVICE_DTYPE.names:
        svc[k] = w.service_columns(1)[k]
    slo = np.zeros(M, tre.SLO_DTYPE)
    for k in tre.SLO_DTYPE.names:
        slo[k] = w.slo_columns(1)[k]
    prof = tre.pack(w.profile_columns(1), tre.PROFILE_DTYPE)
    sc = tre.pack(sc_cols, tre.SCENARIO_DTYPE)
    nW = cfg["duration_ms"] // cfg["window_ms"]
    move_cap = max(1, _n_ticks(cfg) * int(np.max(sc_cols["max_moves"])))
    fp_t = torch.from_numpy(fp).cuda()
    for small in (int(r_init.sum()) - 1, int(r_init.sum())):
        rq, keep = tre.loop_requests(tables, M, svc, slo, r_cap=10, max_replicas=small)
        out = tre.ctl_outputs(_Ev(1, M, nW), 12, move_cap)
        stats = torch.zeros(12 * M * tre.LOOP_STATS_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
        ws = torch.empty(tre.tre_loop_workspace_size(cfg, rq, 12), dtype=torch.uint8, device="cuda")
        tre.tre_loop_act(cfg, 1, rq, prof, sc, tre.actuation(1310, 1870, fp_t), out, stats, ws)
        torch.cuda.synchronize()
        over = int(ws[:8].cpu().numpy().view(np.uint64)[0])
        say(f"bound {small}: {over} counted beyond the declared bounds")
        assert over > 0


def test_argument_errors(lib):
    tre, device, torch = lib
    w = tg.standard(0)
    tables = [w.requests(0)]
    svc = np.zeros(3, tre.SERVICE_DTYPE)
    for k in tre.SERVICE_DTYPE.names:
        svc[k] = w.service_columns(1)[k]
    slo = np.zeros(3, tre.SLO_DTYPE)
    for k in tre.SLO_DTYPE.names:
        slo[k] = w.slo_columns(1)[k]
    cfg = w.trace_cfg()
    rq, keep = tre.loop_requests(tables, 3, svc, slo)
    prof = tre.pack(w.profile_columns(1), tre.PROFILE_DTYPE)
    sc = tre.pack(_scenarios(np.random.default_rng(0), 2, 1), tre.SCENARIO_DTYPE)
    out = tre.ctl_outputs(_Ev(1, 3, 600), 2, 4)
    stats = torch.zeros(2 * 3 * 32, dtype=torch.uint8, device="cuda")
    ws = torch.empty(64, dtype=torch.uint8, device="cuda")
    with pytest.raises(tre.TreError) as e:
        tre.tre_loop(cfg, 1, rq, prof, sc, out, stats, ws)
    assert e.value.code == tre.TRE_ENOMEM
    bad, keep2 = tre.loop_requests(tables, 3, svc, slo, slots_per_replica=0)
    with pytest.raises(tre.TreError) as e:
        tre.tre_loop_workspace_size(cfg, bad, 2)
    assert e.value.code == tre.TRE_EINVAL
    # slot heaps beyond the LDS of one workgroup
    big, keep3 = tre.loop_requests(tables, 3, svc, slo, slots_per_replica=4096, r_cap=4096)
    with pytest.raises(tre.TreError) as e:
        tre.tre_loop_workspace_size(dict(cfg, budget=4096), big, 2)
    assert e.value.code == tre.TRE_EINVAL
    # the actuation model: negative delays
    ws = torch.empty(tre.tre_loop_workspace_size(cfg, rq, 2), dtype=torch.uint8, device="cuda")
    for wake_ms, sleep_ms in ((-1, 0), (0, -250)):
        with pytest.raises(tre.TreError) as e:
            tre.tre_loop_act(cfg, 1, rq, prof, sc, tre.actuation(wake_ms, sleep_ms), out, stats, ws)
        assert e.value.code == tre.TRE_EINVAL
    torch.cuda.synchronize()
