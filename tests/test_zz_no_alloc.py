"""tas_create_static, the entry point for callers that cannot allocate device
memory: the workspace lies in the library's static device array. Its outputs
must equal those of tas_create with a caller-allocated workspace, element by
element, on two calls in a row, the second with a smaller input (the array
keeps the first call's contents)."""
import numpy as np
import pytest

from paper_2606_18431_amd import tas
from paper_2606_18431_amd import workloads as W

pytestmark = pytest.mark.gpu

KEYS = ("ttft", "ttlt", "tbtmax", "counters", "pct", "status")


@pytest.fixture(scope="module")
def torch():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def run_static(torch, w):
    """One step through tas_create_static; host copies of every output."""
    t, keep_t = tas.make_traces(w.arrival_us, w.prompt, w.decode, w.cached)
    p, keep_p = tas.make_params(w.engine, w.settings)
    assert tas.tas_workspace_bytes(t, p) <= tas.STATIC_WORKSPACE_BYTES
    ctx = tas.tas_create_static(t, p)
    try:
        st = torch.cuda.current_stream()
        n, m = w.n_inst, w.n_req
        pct = torch.zeros((n, 3, 3), dtype=torch.int32, device="cuda")
        cnt = torch.zeros((n, 8), dtype=torch.int64, device="cuda")
        status = torch.zeros(n, dtype=torch.int32, device="cuda")
        lat = [torch.empty((n, m), dtype=torch.int32, device="cuda") for _ in range(3)]
        tas.tas_run(ctx, st)
        tas.tas_percentiles(ctx, pct, st)
        tas.tas_latencies(ctx, *lat, stream=st)
        tas.tas_counters(ctx, cnt, st)
        tas.tas_instance_status(ctx, status, st)
        rc = tas.tas_status(ctx)
        torch.cuda.synchronize()
        out = {k: v.cpu().numpy().view(np.uint32) for k, v in zip(KEYS[:3], lat)}
        out.update(counters=cnt.cpu().numpy(), pct=pct.cpu().numpy().view(np.uint32),
                   status=status.cpu().numpy(), rc=rc)
        return out
    finally:
        tas.tas_destroy(ctx)


def run_workspace(w):
    sim = tas.Simulation(w)
    sim.step()
    out = sim.results()
    sim.close()
    return out


def test_static_workspace_equals_caller_workspace(torch):
    # the second call's input is smaller than the first's
    for cfg, n_traces, n_settings, n_req in ((2, 2, 8, 3000), (1, 1, 6, 700)):
        w = W.make(cfg, n_traces=n_traces, n_settings=n_settings, n_req=n_req)
        print(f"[gpu] static workspace: {w.name} {w.n_inst} x {w.n_req}", flush=True)
        a = run_static(torch, w)
        b = run_workspace(w)
        assert a["rc"] == b["rc"] == 0
        for k in KEYS:
            assert np.array_equal(a[k], b[k]), (cfg, k)


def test_static_workspace_rejects_large_inputs():
    w = W.make(4, n_traces=2, n_settings=16)  # 32 x 50,000 requests: beyond the array
    t, keep_t = tas.make_traces(w.arrival_us, w.prompt, w.decode)
    p, keep_p = tas.make_params(w.engine, w.settings)
    assert tas.tas_workspace_bytes(t, p) > tas.STATIC_WORKSPACE_BYTES
    with pytest.raises(tas.TasError) as e:
        tas.tas_create_static(t, p)
    assert e.value.code == tas.TAS_ENOMEM
