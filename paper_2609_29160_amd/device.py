"""Put synthetic workloads (``tracegen``) into HBM for the replay library.

Only data movement lives here: trace columns are generated on the host in
batches of traces into pinned staging buffers and copied into one set of
device columns; profile and scenario tables are packed into the structs of
``include/tre.h``.  No replay arithmetic.
"""
from __future__ import annotations

import time
from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import tre

PAD_ROWS = 16  # rows past the end that stay readable (tile loads round up to 16 bytes)

COLUMNS = (("ts", np.int64, torch.int64), ("model", np.uint8, torch.uint8),
           ("req", np.uint32, torch.uint32), ("type", np.uint8, torch.uint8),
           ("tokens", np.uint16, torch.uint16))


class DeviceTraces:
    """Device columns of traces [t0, t1) of a workload, CSR offsets on the
    host (``off[i]`` = first row of trace t0+i)."""

    def __init__(self, workload, t0, t1, cols, off, counts):
        self.workload = workload
        self.t0, self.t1 = t0, t1
        self.cols = cols
        self.off = off
        self.counts = counts

    @property
    def n_events(self) -> int:
        return int(self.off[-1] - self.off[0])

    @property
    def stored_bytes(self) -> int:
        return sum(v.numel() * v.element_size() for v in self.cols.values())

    def host_trace(self, i: int) -> Dict[str, np.ndarray]:
        """Copy trace t0+i back to the host (for inspection)."""
        a, b = int(self.off[i]), int(self.off[i + 1])
        return {k: v[a:b].cpu().numpy() for k, v in self.cols.items()}


def upload(workload, t0: int = 0, t1: Optional[int] = None, threads: Optional[int] = None,
           batch_events: int = 1 << 28, log=None, keep_host: Sequence[int] = ()) -> DeviceTraces:
    """Generate traces [t0, t1) and copy them into fresh device columns.

    ``keep_host``: indices (relative to t0) whose host columns are returned
    in ``DeviceTraces.host`` (for the CPU checks), without re-generation."""
    import tracegen as tg

    t1 = workload.n_traces if t1 is None else t1
    threads = threads or tg.default_threads()
    t_start = time.time()
    counts = workload.count(t0, t1, threads)
    off = np.zeros(len(counts) + 1, np.int64)
    np.cumsum(counts, out=off[1:])
    total = int(off[-1])
    if log:
        log(f"counted {total} events in {t1 - t0} traces ({time.time() - t_start:.1f} s)")
    # the library reads each column up to 16 bytes past its last row
    cols = {k: torch.zeros(total + PAD_ROWS, dtype=tdt, device="cuda") for k, _, tdt in COLUMNS}
    # pinned staging, reused across batches
    max_batch = max(int(counts.max(initial=0)), min(batch_events, total))
    stage = {k: torch.empty(max(max_batch, 1), dtype=tdt, pin_memory=True) for k, _, tdt in COLUMNS}
    stage_np = {k: stage[k].numpy() for k in stage}
    host = {}
    max_req = -1
    n_arrive = n_finish = 0
    keep = set(int(i) for i in keep_host)
    i = 0
    n = t1 - t0
    while i < n:
        j = i + 1
        while j < n and off[j + 1] - off[i] <= max_batch:
            j += 1
        nb = int(off[j] - off[i])
        ev = workload.generate(t0 + i, t0 + j, threads=threads, out=stage_np, out_offset=0,
                               counts=counts[i:j])
        if nb:
            max_req = max(max_req, int(stage_np["req"][:nb].max()))
            kinds = np.bincount(stage_np["type"][:nb] & 3, minlength=4)
            n_arrive += int(kinds[0])
            n_finish += int(kinds[3])
        for k in cols:
            cols[k][int(off[i]):int(off[j])].copy_(stage[k][:nb], non_blocking=True)
        for r in range(i, j):
            if r in keep:
                a, b = int(off[r] - off[i]), int(off[r + 1] - off[i])
                host[r] = {k: stage_np[k][a:b].copy() for k in stage_np}
        torch.cuda.current_stream().synchronize()  # staging is reused next batch
        del ev
        if log:
            log(f"uploaded traces [{t0 + i}, {t0 + j}) ({off[j]} events, {time.time() - t_start:.1f} s)")
        i = j
    dt = DeviceTraces(workload, t0, t1, cols, off, counts)
    dt.host = host
    dt.req_cap = max_req + 1  # request ids of every trace are below this
    dt.n_arrive, dt.n_finish = n_arrive, n_finish
    return dt


def load(dt: DeviceTraces, validate: bool = True, budget: Optional[int] = None) -> tre.Events:
    """budget: replaces the workload's budget (GPUs under the actuation model)."""
    c = dt.cols
    cfg = dict(dt.workload.trace_cfg())
    if budget is not None:
        cfg["budget"] = int(budget)
    return tre.tre_load_events(c["ts"], c["model"], c["req"], c["type"], c["tokens"], dt.off, cfg,
                               validate=validate)


def profiles(workload, n_traces: Optional[int] = None) -> torch.Tensor:
    return tre.pack(workload.profile_columns(n_traces), tre.PROFILE_DTYPE)


def slos(workload, n_traces: Optional[int] = None) -> torch.Tensor:
    return tre.pack(workload.slo_columns(n_traces), tre.SLO_DTYPE)


def scenarios(cols: Dict[str, np.ndarray]) -> torch.Tensor:
    return tre.pack(cols, tre.SCENARIO_DTYPE)
