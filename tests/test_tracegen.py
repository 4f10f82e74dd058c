"""The synthetic workload generator: determinism, schema, lifecycle, sizes."""
import numpy as np
import pytest

import tracegen as tg


def _lifecycle_ok(ev, M, duration_ms):
    ts, model, typ, req = ev["ts"], ev["model"], ev["type"], ev["req"]
    assert np.all(np.diff(ts) >= 0)
    assert ts.min() >= 0 and ts.max() < duration_ms
    assert model.max() < M
    kind = typ & 3
    admit = (typ & 0x80) != 0
    assert np.all((typ & 0x7C) == 0)
    assert np.all(kind[admit] == 1)
    # per-model running counts never negative
    dW = np.where(kind == 0, 1, 0) - np.where(admit, 1, 0)
    dA = np.where(admit, 1, 0) - np.where(kind == 3, 1, 0)
    for m in range(M):
        sel = model == m
        assert np.cumsum(dW[sel]).min(initial=0) >= 0
        assert np.cumsum(dA[sel]).min(initial=0) >= 0
    # each request: one ARRIVE first, at most one ADMIT, FINISH last
    order = np.lexsort((np.arange(len(req)), req))
    r, k, a = req[order], kind[order], admit[order]
    starts = np.r_[True, r[1:] != r[:-1]]
    assert np.all(k[starts] == 0)
    ends = np.r_[r[1:] != r[:-1], True]
    fin = k == 3
    assert np.all(ends[fin])
    n_admit = np.bincount(np.searchsorted(r[starts], r), weights=a.astype(np.int64))
    assert n_admit.max() <= 1
    tok = ev["tokens"]
    assert np.all(tok[kind == 1] <= 2048) and np.all(tok[kind == 2] <= 24) and np.all(tok[kind == 3] == 0)


@pytest.mark.parametrize("i", [0, 1])
def test_schema_and_lifecycle(i):
    w = tg.standard(i)
    ev = w.generate(0, 1, threads=4).trace(0)
    _lifecycle_ok(ev, w.n_models, w.duration_ms)


@pytest.mark.parametrize("i", [3, 4])
def test_schema_and_lifecycle_short(i):
    w = tg.standard(i).scaled(duration_ms=300_000, n_traces=3)
    evs = w.generate(0, 3, threads=4)
    for t in range(3):
        _lifecycle_ok(evs.trace(t), w.n_models, w.duration_ms)


def test_deterministic_and_batch_independent():
    w = tg.standard(4).scaled(duration_ms=120_000, n_traces=5)
    a = w.generate(0, 5, threads=1)
    b = w.generate(0, 5, threads=4)
    c = w.generate(2, 4, threads=2)
    for k in ("ts", "model", "req", "type", "tokens"):
        assert np.array_equal(a[k], b[k])
        assert np.array_equal(a.trace(2)[k], c.trace(0)[k])
        assert np.array_equal(a.trace(3)[k], c.trace(1)[k])
    # different traces differ
    assert not np.array_equal(a.trace(0)["ts"][:100], a.trace(1)["ts"][:100])


def test_generate_into_preallocated_columns():
    w = tg.standard(0)
    n = int(w.count().sum())
    cols = {"ts": np.zeros(n + 10, np.int64), "model": np.zeros(n + 10, np.uint8),
            "req": None, "type": np.zeros(n + 10, np.uint8), "tokens": np.zeros(n + 10, np.uint16)}
    ev = w.generate(out=cols, out_offset=10)
    ref = w.generate()
    assert ev.off[0] == 10 and ev.off[-1] == n + 10
    assert np.array_equal(cols["ts"][10:], ref["ts"])


def test_sizes_match_workload_shapes():
    # events per workload near the advertised shapes (about 50k, 2M, 1.5e9,
    # and 150 GB at 16 bytes per stored event)
    n0 = int(tg.standard(0).count().sum())
    assert 40_000 < n0 < 60_000
    n1 = int(tg.standard(1).count().sum())
    assert 1.6e6 < n1 < 2.4e6
    w3 = tg.standard(3)
    est3 = tg.standard(3).count(0, 2).mean() * w3.n_traces
    assert 1.2e9 < est3 < 1.8e9
    w4 = tg.standard(4)
    est4 = w4.count(0, 4).mean() * w4.n_traces
    assert 120e9 < est4 * 16 < 180e9


def test_scenario_tables():
    s2 = tg.standard(2).scenario_columns()
    assert s2["trace"].shape == (1024,) and np.all(s2["trace"] == 0)
    assert np.all((s2["theta_scale"] >= 0.5) & (s2["theta_scale"] <= 2.0))
    assert set(np.unique(s2["max_moves"]).tolist()) == {1, 2, 4}
    assert np.all((s2["tau_crit_override"] >= 0.2) & (s2["tau_crit_override"] <= 0.8))
    s4 = tg.standard(4).scenario_columns()
    assert np.array_equal(s4["trace"], np.arange(4096))
    s0 = tg.standard(0).scenario_columns()
    assert s0["max_moves"][0] == 1 and s0["tau_crit_override"][0] < 0
