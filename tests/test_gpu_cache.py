"""Parity of the cache-aware boost signal (paper: interaction with
prefix/radix caching; the signal P - h + dec with h expected cached prompt
tokens) on the GPU with the CPU oracle, through the C ABI. Element by element
and exact: the cache-aware settings beside the plain signal, FCFS and SRPT in
one launch; with the on-chip list cut to its minimum (spills, refills, the
retry pass); combined with adaptive gamma; and at the extremes of the hits
(none, and all but one prompt token)."""
import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def gpu_run(w, **kw):
    from paper_2606_18431_amd import tas

    print(f"[gpu] {w.name} cache traces={w.n_traces} inst={w.n_inst} n_req={w.n_req} {kw}",
          flush=True)
    sim = tas.Simulation(w, **kw)
    sim.step()
    out = sim.results()
    sim.close()
    return out


def assert_parity(g, o):
    assert np.array_equal(g["status"], o["status"]), (g["status"], o["status"])
    assert np.all(g["status"] == 0)
    for key in ("ttft", "ttlt", "tbtmax", "counters", "pct", "switches"):
        if not np.array_equal(g[key], o[key]):
            bad = np.argwhere(g[key] != o[key])[0]
            raise AssertionError(f"{key} differs first at {tuple(bad)}: gpu {g[key][tuple(bad)]} "
                                 f"oracle {o[key][tuple(bad)]}")
    assert np.array_equal(g["gamma"].view(np.int64), o["gamma"].view(np.int64))


@pytest.mark.parametrize("cfg,n_traces,n_req", [(1, 2, 3000), (2, 2, 3000), (3, 1, 5000),
                                                (0, 1, 1000)])
def test_parity_cache_grid(torch, cfg, n_traces, n_req):
    w = W.make(cfg, n_traces=n_traces, n_req=n_req, grid="cache")
    g = gpu_run(w)
    o = oracle.run(w)
    assert_parity(g, o)


@pytest.mark.parametrize("cfg,extra", [(2, 0), (3, 64)])
def test_parity_cache_with_spill(torch, cfg, extra):
    w = W.make(cfg, n_traces=1, n_req=3000, grid="cache")
    g = gpu_run(w, list_cap=w.engine.max_seqs + 64 + extra)
    o = oracle.run(w)
    assert_parity(g, o)


def test_parity_cache_with_adaptive_gamma(torch):
    """The cache-aware signal under adaptive gamma (every grid change re-keys
    by the stored level, which follows P - h + dec), beside the ladder."""
    base = W.make(2, n_traces=1, n_req=3000, grid="ladder")
    extra = [W.setting(0, W.BOOST, gamma=1e-3, signal=2, ada=dict(W.ADA, window=40,
                                                                 min_samples=20), **W.UNIBOOST),
             W.setting(0, W.BOOST, gamma=1e-2, signal=2, ada=dict(W.ADA), **W.VANILLA)]
    sets = np.concatenate([base.settings, np.stack(extra)])
    h = W.cached_tokens([2, 0], base.prompt[0])[None]
    w = W.Workload(base.name, base.arrival_us, base.prompt, base.decode, base.engine, sets,
                   cached=h)
    g = gpu_run(w)
    o = oracle.run(w)
    assert_parity(g, o)
    assert np.all(o["switches"][-2:] > 0)


def test_parity_cache_extremes(torch):
    """Hits of 0 (the plain signal) and P - 1 (one prompt token of work) on
    two traces, and the cache-aware signal differs from the plain one."""
    base = W.make(1, n_traces=2, n_req=3000, grid="cache")
    h = np.stack([np.zeros_like(base.prompt[0]), base.prompt[1] - 1]).astype(np.int32)
    w = W.Workload(base.name, base.arrival_us, base.prompt, base.decode, base.engine,
                   base.settings, cached=h)
    g = gpu_run(w)
    o = oracle.run(w)
    assert_parity(g, o)
    for i in range(0, 6, 2):
        assert np.array_equal(g["ttlt"][i], g["ttlt"][i + 1])  # no hits: same schedule
        assert not np.array_equal(g["ttlt"][8 + i], g["ttlt"][8 + i + 1])
