"""Shared helpers of the GPU parity tests: run the HIP library and the CPU
oracle on the same seeded inputs and compare.

Bars: integer tallies, flags, move logs, final replicas and replica-window
sums bit-exact; the fp64 smoothed TSS bit-exact (the decisions compare it);
the fp32 TSS within 1e-5 relative of the oracle's fp64 value (and equal to
its round-to-nearest fp32 conversion).
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np

import oracle as O

TSS_REL_TOL = 1e-5


def oracle_tss(host: Dict[str, np.ndarray], workload, prof_cols_trace) -> Dict[str, np.ndarray]:
    prof = O.pack_profiles(prof_cols_trace)
    return O.get().tss_trace(host, workload.window_ms, workload.duration_ms, prof)


def compare_tss(gpu: Dict[str, np.ndarray], ref: Dict[str, np.ndarray], what: str):
    """gpu: per-cell arrays [n_windows][M] of one trace; ref: oracle dict."""
    assert np.array_equal(gpu["prefill"].astype(np.int64), ref["P"]), f"{what}: prefill tokens"
    assert np.array_equal(gpu["decode"].astype(np.int64), ref["D"]), f"{what}: decode tokens"
    assert np.array_equal(gpu["a_int"], ref["A_int"]), f"{what}: active integral"
    assert np.array_equal(gpu["w_int"], ref["W_int"]), f"{what}: waiting integral"
    assert np.array_equal(gpu["flags"], ref["flags"]), f"{what}: flags"
    s64 = gpu["tss64"]
    bad = np.flatnonzero(s64.view(np.int64) != ref["S"].view(np.int64))
    assert bad.size == 0, f"{what}: fp64 TSS differs at {bad[:5]} ({s64.reshape(-1)[bad[:5]]} vs {ref['S'].reshape(-1)[bad[:5]]})"
    compare_tss32(gpu["tss32"], ref["S"], what)


FLT_MIN = 2.0 ** -126


def compare_tss32(t32: np.ndarray, s64: np.ndarray, what: str):
    """fp32 TSS: within 1e-5 relative of the oracle's fp64 value wherever that
    value is in fp32's normal range; below it (values decaying towards zero
    through smoothing) within half a subnormal step; and in both cases equal
    to the round-to-nearest fp32 conversion."""
    ref = s64.astype(np.float64)
    got = t32.astype(np.float64)
    normal = np.abs(ref) >= FLT_MIN
    rel = np.abs(got - ref)[normal] / np.abs(ref)[normal]
    assert rel.size == 0 or rel.max() <= TSS_REL_TOL, f"{what}: fp32 TSS off by {rel.max():.3g} relative"
    tiny = np.abs(got - ref)[~normal]
    assert tiny.size == 0 or tiny.max() <= 2.0 ** -150, f"{what}: subnormal fp32 TSS off by {tiny.max():.3g}"
    rn = s64.astype(np.float32)
    bad = np.flatnonzero(t32.view(np.uint32) != rn.view(np.uint32))
    assert bad.size == 0, f"{what}: fp32 TSS is not the RN conversion at {bad[:5]}: {t32.reshape(-1)[bad[:5]]} vs {rn.reshape(-1)[bad[:5]]}"


def compare_ctl(moves: np.ndarray, n_moves: int, r_final, r_windows, ref, what: str):
    assert n_moves == ref["n_moves"], f"{what}: {n_moves} moves vs {ref['n_moves']}"
    k = min(n_moves, len(moves))
    got = moves[:k]
    exp = ref["moves"][:k]
    for f in ("window", "path", "receiver", "donor"):
        assert np.array_equal(got[f], exp[f]), f"{what}: move {f} differs"
    assert np.array_equal(np.asarray(r_final), ref["r_final"]), f"{what}: final replicas"
    assert np.array_equal(np.asarray(r_windows), ref["r_windows"]), f"{what}: replica-window sums"


def oracle_control(workload, prof_cols_trace, S, flags, sc_row, move_cap: Optional[int] = None):
    prof = O.pack_profiles(prof_cols_trace)
    sc = np.zeros(1, O.SCENARIO_DTYPE)
    for k in O.SCENARIO_DTYPE.names:
        sc[k] = sc_row[k]
    return O.get().control(workload.trace_cfg(), prof, S, flags, sc, move_cap)


def trace_profile(prof_cols, t, M):
    return {k: v[t * M:(t + 1) * M] for k, v in prof_cols.items()}
