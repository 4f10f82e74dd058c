"""tre_sweep_noalloc: the sweep with its scratch in the library's static
device array, for callers that cannot allocate. Through the C ABI, two calls
in a row (the second on a smaller input) must give exactly the outputs of
tre_sweep on the same inputs (move logs, move counts, final replicas,
replica-window sums, per-cell fp32 TSS), and a sweep whose scratch exceeds
the static array must be refused with TRE_ENOMEM."""
import sys

import numpy as np
import pytest

import tracegen as tg

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _host(o):
    from paper_2609_29160_amd import tre
    return {"moves": tre.unpack_moves(o["moves"]).copy(), "n_moves": o["n_moves"].cpu().numpy(),
            "r_final": o["r_final"].cpu().numpy(), "r_windows": o["r_windows"].cpu().numpy()}


def _compare_one(w, n_traces):
    import torch

    from paper_2609_29160_amd import device, tre

    w = w.scaled(n_traces=n_traces, n_scenarios=n_traces)
    dt = device.upload(w)
    ev = device.load(dt)
    prof = device.profiles(w)
    sc_cols = w.scenario_columns()
    sc = device.scenarios(sc_cols)
    n_sc = len(sc_cols["trace"])
    cap = ev.n_ticks * int(np.max(sc_cols["max_moves"]))
    need = tre.tre_workspace_size(ev, n_sc)
    say(f"{w.name}: {n_traces} traces, {dt.n_events} events, scratch {need} bytes")
    assert need <= tre.TRE_NOALLOC_SCRATCH_BYTES
    ref = tre.ctl_outputs(ev, n_sc, cap)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    t32_ref = torch.empty((ev.n_traces, ev.n_windows, ev.n_models), dtype=torch.float32, device="cuda")
    tre.tre_sweep(ev, prof, sc, ref, ws, tss32=t32_ref)
    got = tre.ctl_outputs(ev, n_sc, cap)
    t32 = torch.full_like(t32_ref, -1.0)
    tre.tre_sweep_noalloc(ev, prof, sc, got, tss32=t32)
    torch.cuda.synchronize()
    a, b = _host(ref), _host(got)
    for k in a:
        assert np.array_equal(np.asarray(a[k]).view(np.uint8), np.asarray(b[k]).view(np.uint8)), f"{w.name}: {k}"
    assert torch.equal(t32_ref.view(torch.int32), t32.view(torch.int32)), f"{w.name}: tss32"
    moved = int((a["n_moves"] > 0).sum())
    say(f"{w.name}: equal to tre_sweep ({moved} of {n_sc} scenarios with moves)")
    ev.close()


def test_noalloc_equals_sweep_twice():
    """A 48-trace diverse-shaped input (16 models, 7200 windows: 8.8 MB of
    scratch), then a smaller one (the 3-model workload, one trace)."""
    from paper_2609_29160_amd import tre
    assert tre.TRE_NOALLOC_SCRATCH_BYTES == 64 << 20
    _compare_one(tg.standard(3), 48)
    _compare_one(tg.standard(0), 1)


def test_noalloc_refuses_too_large():
    """4096 traces x 32 models x 720 ticks need 755 MB of scratch: refused
    before any launch (empty traces, so no events are needed)."""
    import torch

    from paper_2609_29160_amd import tre

    w = tg.standard(4)
    cfg = w.trace_cfg()
    cols = {k: torch.zeros(16, dtype=d, device="cuda") for k, d in
            (("ts", torch.int64), ("model", torch.uint8), ("req", torch.uint32), ("type", torch.uint8),
             ("tokens", torch.uint16))}
    off = np.zeros(4097, np.int64)
    ev = tre.tre_load_events(cols["ts"], cols["model"], cols["req"], cols["type"], cols["tokens"], off, cfg)
    prof = tre.pack(w.profile_columns(), tre.PROFILE_DTYPE)
    sc = tre.pack(w.scenario_columns(), tre.SCENARIO_DTYPE)
    out = tre.ctl_outputs(ev, 4096, 4)
    with pytest.raises(tre.TreError) as e:
        tre.tre_sweep_noalloc(ev, prof, sc, out)
    assert e.value.code == tre.TRE_ENOMEM, str(e.value)
    say("too large:", e.value)
    ev.close()
