"""GPU parity of the stage-aware service shares against the oracle's, by
both paths: tre_stage_tss (from the tallies of tre_eval_tss) and
tre_eval_stage (one pass over the events).

For every trace: the per-window prefill and decode shares in binary64 bit
for bit, their binary32 copies equal to the round-to-nearest conversion of
the oracle's values (hence within 1e-5 relative), and the flags exactly.
The tallies fed to tre_stage_tss are tre_eval_tss's (themselves compared
with the oracle's in the main parity tests); the oracle computes its shares
from its own tallies.

Inputs: the tiny and bursty workloads whole, short diverse and stress
traces (many windows, ragged ends), the hand-built trace of the oracle's
pins, a decode-only trace, empty / sparse / boundary / dense-window edge
traces, 1 / 17 / 64 models, window widths 1 ms to 60 s, launch-to-launch
determinism and argument errors.
"""
import sys

import numpy as np
import pytest

import oracle as O
import parity as PT
import stage_pins as SP
import edge_traces as E
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


def _cfg(M, win, nW):
    return {"window_ms": win, "duration_ms": win * nW, "fast_period_ms": win, "slow_period_ms": 2 * win,
            "n_models": M, "budget": 2 * M}


def _check(lib, name, cfg, traces, prof_cols, repeat=1):
    tre, device, torch = lib
    M, win, dur = cfg["n_models"], cfg["window_ms"], cfg["duration_ms"]
    cols, off = _columns(torch, traces)
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
    prof = tre.pack(prof_cols, tre.PROFILE_DTYPE)
    tal = tre.tss_outputs(ev, which=("prefill", "decode", "a_int", "w_int"))
    tre.tre_eval_tss(ev, prof, tal)
    results = {}
    for path in ("two-pass", "fused"):
        for _ in range(repeat):
            out = tre.stage_outputs(ev)
            if path == "two-pass":
                tre.tre_stage_tss(ev, prof, tal, out)
            else:
                tre.tre_eval_stage(ev, prof, out)
            torch.cuda.synchronize()
            got = {k: v.cpu().numpy() for k, v in out.items()}
            if path not in results:
                results[path] = got
            else:
                for k in got:
                    assert np.array_equal(got[k].view(np.uint8), results[path][k].view(np.uint8)), \
                        f"{name}: {path} {k} differs between launches"
    o = O.get()
    for t, tr in enumerate(traces):
        p = PT.trace_profile(prof_cols, t, M)
        ref_t = o.tss_trace(tr, win, dur, O.pack_profiles(p))
        ref = o.stage_tss(ref_t, win, O.pack_profiles(p))
        for path, first in results.items():
            what = f"{name} trace {t} ({path})"
            s64 = first["stage64"][t]
            bad = np.flatnonzero(s64.view(np.uint64) != ref["S"].view(np.uint64))
            assert bad.size == 0, f"{what}: binary64 shares differ at {bad[:5]}: {s64.reshape(-1)[bad[:5]]} vs {ref['S'].reshape(-1)[bad[:5]]}"
            for k, stage in ((0, "prefill"), (1, "decode")):
                PT.compare_tss32(first["stage32"][t][..., k], ref["S"][..., k], f"{what} {stage} binary32")
            assert np.array_equal(first["flags"][t], ref["flags"]), f"{what}: flags"
    ev.close()


def _workload(lib, name, w, n):
    w = w.scaled(n_traces=n) if w.n_traces != n else w
    evs = w.generate(0, n, threads=8)
    traces = [evs.trace(i) for i in range(n)]
    say(f"{name}: {sum(len(t['ts']) for t in traces)} events")
    _check(lib, name, w.trace_cfg(), traces, w.profile_columns(n))


def test_tiny(lib):
    _workload(lib, "tiny", tg.standard(0), 1)


def test_bursty(lib):
    _workload(lib, "bursty", tg.standard(1), 1)


def test_diverse_short(lib):
    _workload(lib, "diverse", tg.standard(3).scaled(duration_ms=1_200_000), 3)


def test_stress_short(lib):
    _workload(lib, "stress", tg.standard(4).scaled(duration_ms=900_000), 5)


def _rand_prof(M, n, seed):
    rng = np.random.default_rng(seed)
    k = M * n
    return {"w_p": rng.uniform(0.05, 0.9, k), "w_q": rng.uniform(1.0, 3.0, k), "alpha": rng.uniform(0.05, 1.0, k),
            "theta": rng.uniform(1, 100, k), "tau_crit": rng.uniform(0.2, 0.6, k),
            "tau_surplus": rng.uniform(1.1, 2.0, k), "r_min": np.zeros(k, np.int32), "r_init": np.ones(k, np.int32)}


def test_hand_and_decode_only(lib):
    """The oracle pins' hand trace (w_p 1/2, w_q 2, alpha 1/2) and a trace
    with empty prompts admitted on arrival."""
    rows = [(0, 0, 0, 0, 100), (700, 0, 0, 0x81, 100), (800, 0, 0, 2, 24), (1200, 0, 0, 2, 24), (1500, 0, 0, 3, 0),
            (1000, 0, 1, 0, 50), (1000, 0, 1, 0x81, 50), (1600, 0, 1, 2, 24), (2300, 0, 1, 2, 12), (2300, 0, 1, 3, 0),
            (3000, 0, 2, 0, 10), (100, 1, 3, 0, 3000), (200, 1, 3, 0x81, 3000), (900, 1, 3, 3, 0)]
    rows.sort(key=lambda r: (r[0], r[3] & 3))
    hand = SP._trace(rows)
    p = SP._prof(2)
    cols = {k: np.array([p[k][0]] * 2) for k in O.PROFILE_DTYPE.names}
    _check(lib, "hand", _cfg(2, 1000, 4), [hand], cols)
    rng = np.random.default_rng(11)
    rows = []
    for rid in range(300):
        m = int(rng.integers(0, 3))
        t = int(rng.integers(0, 500_000))
        rows += [(t, m, rid, 0, 0), (t, m, rid, 0x81, 0)]
        for _ in range(int(rng.integers(1, 6))):
            t += int(rng.integers(1, 4000))
            rows.append((t, m, rid, 2, int(rng.integers(1, 25))))
        rows.append((t, m, rid, 3, 0))
    done = {r[2] for r in rows if r[3] == 3 and r[0] < 600_000}
    rows = sorted([r for r in rows if r[2] in done], key=lambda r: (r[0], r[3] & 3))
    _check(lib, "decode-only", _cfg(3, 1000, 600), [SP._trace(rows)], _rand_prof(3, 1, 4))


def test_edge_traces(lib):
    M, win, nW = 8, 100, 3000
    traces = [E.trace_random(1, M, win * nW, 3000), E.trace_empty(), E.trace_sparse(2, M, win, nW, gap_windows=700),
              E.trace_boundaries(M, win, nW), E.trace_dense_window(M, win, nW, 1234, 60000),
              E.trace_identical_models(M, win, nW), E.trace_empty()]
    _check(lib, "edge", _cfg(M, win, nW), traces, _rand_prof(M, len(traces), 7), repeat=2)


@pytest.mark.parametrize("M", [1, 17, 64])
def test_model_counts(lib, M):
    win, nW = 250, 2400
    traces = [E.trace_random(10 + M + i, M, win * nW, 400 * M) for i in range(3)]
    _check(lib, f"M{M}", _cfg(M, win, nW), traces, _rand_prof(M, 3, M))


@pytest.mark.parametrize("win", [1, 7, 60000])
def test_window_widths(lib, win):
    M = 5
    nW = max(8, min(20000, 3_600_000 // win))
    traces = [E.trace_random(20 + i, M, win * nW, 3000) for i in range(2)]
    _check(lib, f"win{win}", _cfg(M, win, nW), traces, _rand_prof(M, 2, win))


def test_argument_errors(lib):
    tre, device, torch = lib
    M, win, nW = 3, 100, 50
    cfg = _cfg(M, win, nW)
    cols, off = _columns(torch, [E.trace_random(3, M, win * nW, 200)])
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
    prof = tre.pack(_rand_prof(M, 1, 0), tre.PROFILE_DTYPE)
    tal = tre.tss_outputs(ev, which=("prefill", "decode", "a_int", "w_int"))
    tre.tre_eval_tss(ev, prof, tal)
    out = tre.stage_outputs(ev)
    with pytest.raises(tre.TreError) as e:
        tre.tre_stage_tss(ev, prof, {k: v for k, v in tal.items() if k != "w_int"}, out)
    assert e.value.code == tre.TRE_EINVAL
    with pytest.raises(tre.TreError) as e:
        tre.tre_stage_tss(ev, prof, tal, {})
    assert e.value.code == tre.TRE_EINVAL
    bad = torch.empty(2 * M * nW * 2 + 1, dtype=torch.float64, device="cuda")[1:]
    with pytest.raises(tre.TreError) as e:
        tre.tre_stage_tss(ev, prof, tal, {"stage64": bad})
    assert e.value.code == tre.TRE_EINVAL
    for o in ({}, {"stage64": bad}):
        with pytest.raises(tre.TreError) as e:
            tre.tre_eval_stage(ev, prof, o)
        assert e.value.code == tre.TRE_EINVAL
    torch.cuda.synchronize()
    ev.close()
