"""Small hand-shaped traces for edge cases (inputs only, no TSS arithmetic).

Each function returns host columns sorted by ts with equal timestamps in
lifecycle order, so the active / waiting counts never go negative.
"""
from __future__ import annotations

import numpy as np


def _pack(rows):
    if not rows:
        z = lambda dt: np.zeros(0, dt)
        return {"ts": z(np.int64), "model": z(np.uint8), "req": z(np.uint32), "type": z(np.uint8),
                "tokens": z(np.uint16)}
    a = np.array(rows, dtype=np.int64)
    order = np.lexsort((np.arange(len(a)), a[:, 0]))  # stable by ts
    a = a[order]
    return {"ts": a[:, 0].astype(np.int64), "model": a[:, 1].astype(np.uint8),
            "req": a[:, 2].astype(np.uint32), "type": a[:, 3].astype(np.uint8),
            "tokens": a[:, 4].astype(np.uint16)}


def random_requests(rng, M, duration_ms, n_req, t_lo=0, t_hi=None, model_weights=None,
                    admit_p=0.85, finish_p=0.8, max_span_ms=None):
    """Random lifecycle-valid requests: ARRIVE, maybe ADMIT (+ more prefill
    chunks and decodes), maybe FINISH, all inside [t_lo, t_hi)."""
    t_hi = duration_ms if t_hi is None else t_hi
    span = max_span_ms or max(1, (t_hi - t_lo) // 4)
    rows = []
    for r in range(n_req):
        m = int(rng.choice(M, p=model_weights)) if model_weights is not None else int(rng.integers(M))
        a = int(rng.integers(t_lo, t_hi))
        rows.append((a, m, r, 0, int(rng.integers(16, 4000))))
        if rng.random() > admit_p:
            continue
        s = min(t_hi - 1, a + int(rng.integers(0, span)))
        n_pf = int(rng.integers(1, 3))
        t = s
        for k in range(n_pf):
            rows.append((t, m, r, 1 | (0x80 if k == 0 else 0), int(rng.integers(1, 2049))))
            t = min(t_hi - 1, t + int(rng.integers(0, 50)))
        n_dec = int(rng.integers(0, 6))
        for _ in range(n_dec):
            t = min(t_hi - 1, t + int(rng.integers(0, span // 4 + 1)))
            rows.append((t, m, r, 2, int(rng.integers(1, 25))))
        if rng.random() < finish_p:
            rows.append((t, m, r, 3, 0))
    return rows


def trace_random(seed, M, duration_ms, n_req, **kw):
    rng = np.random.default_rng(seed)
    return _pack(random_requests(rng, M, duration_ms, n_req, **kw))


def trace_empty():
    return _pack([])


def trace_boundaries(M, window_ms, n_windows):
    """Every event on an exact window boundary."""
    rows = []
    r = 0
    for w in range(n_windows - 1):
        t = w * window_ms
        m = w % M
        rows += [(t, m, r, 0, 5), (t, m, r, 0x81, 5), (t + window_ms, m, r, 2, 7), (t + window_ms, m, r, 3, 0)]
        r += 1
    return _pack(rows)


def trace_sparse(seed, M, window_ms, n_windows, gap_windows):
    """Short bursts separated by long idle gaps (more windows than the LDS
    ring holds), plus a late first event."""
    rng = np.random.default_rng(seed)
    rows = []
    r0 = 0
    t = gap_windows * window_ms + 3
    dur = n_windows * window_ms
    while t < dur:
        hi = min(dur, t + 3 * window_ms)
        reqs = random_requests(rng, M, dur, 20, t_lo=t, t_hi=hi, max_span_ms=window_ms)
        rows += [(a, m, r + r0, k, tok) for (a, m, r, k, tok) in reqs]
        r0 += 20
        t = hi + gap_windows * window_ms
    return _pack(rows)


def trace_dense_window(M, window_ms, n_windows, w_dense, n_events):
    """n_events / 2 requests of one model arriving and admitted inside one
    window (plus a little background)."""
    rows = []
    base = w_dense * window_ms
    for r in range(n_events // 2):
        t = base + (r * window_ms) // (n_events // 2)
        rows += [(t, 0, r, 0, 10), (t, 0, r, 0x81, 10)]
    return _pack(rows)


def trace_identical_models(M, window_ms, n_windows):
    """Every model gets exactly the same events: every Z ties."""
    rng = np.random.default_rng(3)
    base = random_requests(rng, 1, n_windows * window_ms, 40)
    rows = []
    for m in range(M):
        rows += [(a, m, r * M + m, k, tok) for (a, _, r, k, tok) in base]
    return _pack(rows)
