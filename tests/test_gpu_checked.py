"""The checking build (libtas_check.so) on the GPU.

It runs the same kernels as libtas.so and, after every simulated iteration
of every instance, verifies the state: the batch respects the sequence cap,
the token budget and the KV budget; the list's residents, waiting entries
and holes match their counts; the KV in use is the residents' blocks; the
keys of the live entries ascend strictly; no mark of an iteration survives
it; every spilled entry is waiting and the spill's minimum is exact; every
request taken is done, on chip or spilled. A violation fails the instance
with TAS_ESTATE. Each workload below must finish with no violation and with
the ordinary build's outputs, byte for byte. The workloads cover the spill
and refill paths (the smallest lists), the retry pass, evictions under KV
pressure, every comparator, adaptive gamma, the phase ladder, the
cache-aware signal and the JSQ router; and every full-size workload with
stored oracle digests (configs 1-3, the large sweep and its other settings
grids, the starvation mix), checked against those digests.
"""
import os

import numpy as np
import pytest

from paper_2606_18431_amd import workloads as W

pytestmark = pytest.mark.gpu

SMALL_ADA = [dict(W.ADA, window=24, min_samples=20, beta=0.05, grid=41),
             dict(W.ADA, window=64, min_samples=64, beta=1.0, grid=64, gamma_min=1e-4,
                  gamma_max=3e-1)]
JSQ_SETS = [dict(policy=W.FCFS), dict(policy=W.SRPT), dict(policy=W.BOOST, gamma=1e-3, **W.UNIBOOST),
            dict(policy=W.SARATHI), dict(policy=W.DIST, gamma=1e-3), dict(policy=W.LAS)]


@pytest.fixture(scope="module")
def torch():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def ada_workload(cfg, n_req):
    base = W.make(cfg, n_traces=1, n_req=n_req)
    sets = [W.setting(0, W.BOOST, gamma=1e-3, ada=a, **(W.UNIBOOST if i % 2 == 0 else W.VANILLA))
            for i, a in enumerate(SMALL_ADA)]
    return W.Workload(base.name + " adaptive", base.arrival_us, base.prompt, base.decode,
                      base.engine, np.stack(sets))


def residents_burst_workload(n=200):
    """Everyone arrives at once under a least-attained-service table: old
    residents pause behind fresh arrivals, so more requests hold KV than
    max_seqs and a small list sends the instance to the retry pass."""
    tb = [(23 - j) * 10 ** 11 for j in range(24)]
    e = W.Engine(max_seqs=8, kv_blocks=4096, chunk=64, max_tokens=512)
    sets = np.stack([W.setting(0, W.BOOST, k=1, table=tb), W.setting(0, W.FCFS)])
    return W.Workload("residents burst", np.zeros((1, n), np.int64), np.ones((1, n), np.int32),
                      np.full((1, n), 50, np.int32), e, sets)


def case(name):
    """(workload, Simulation keyword arguments) of the named case."""
    if name == "config0":
        return W.make(0), {}
    if name == "kv-pressure-minimum-list":
        return W.make(2, n_traces=1, n_settings=8, n_req=4000), dict(list_cap=128)
    if name == "bursty-spill":
        return W.make(3, n_traces=1, n_settings=8, n_req=4000), dict(list_cap=128)
    if name == "comparators-spill":
        w = W.make(3, n_traces=1, n_req=4000, grid="comparators")
        return w, dict(list_cap=w.engine.max_seqs + 64)
    if name == "adaptive-gamma-spill":
        w = ada_workload(2, 3000)
        return w, dict(list_cap=w.engine.max_seqs + 64)
    if name == "ladder-spill":
        w = W.make(2, n_traces=1, n_req=3000, grid="ladder")
        return w, dict(list_cap=w.engine.max_seqs + 64)
    if name == "cache-spill":
        w = W.make(3, n_traces=1, n_req=3000, grid="cache")
        return w, dict(list_cap=w.engine.max_seqs + 128)
    if name == "jsq":
        return W.make_cluster(2, n_clusters=1, replicas=4, dispatch="jsq", n_req=300,
                              settings=JSQ_SETS), {}
    if name == "residents-retry":
        return residents_burst_workload(), dict(list_cap=72)
    if name == "large-sweep-law":
        return W.make(4, n_traces=1, n_settings=16, n_req=20000), {}
    raise KeyError(name)


CASES = ["config0", "kv-pressure-minimum-list", "bursty-spill", "comparators-spill",
         "adaptive-gamma-spill", "ladder-spill", "cache-spill", "jsq", "residents-retry",
         "large-sweep-law"]


def run_with(path, w, kw):
    from paper_2606_18431_amd import tas

    prev = tas.select_library(path)
    try:
        sim = tas.Simulation(w, **kw)
        sim.step()
        out = sim.results()
        sim.close()
    finally:
        tas.select_library(prev)
    return out


@pytest.mark.parametrize("name", CASES)
def test_checking_build_finds_no_violation(torch, name):
    from paper_2606_18431_amd import tas

    assert os.path.exists(tas.CHECK_LIB_PATH), "libtas_check.so is missing: run the build"
    w, kw = case(name)
    print(f"[gpu] checked {name}: inst={w.n_inst} n_req={w.n_req} {kw}", flush=True)
    plain = run_with(tas.LIB_PATH, w, kw)
    checked = run_with(tas.CHECK_LIB_PATH, w, kw)
    assert not np.any(checked["status"] == tas.TAS_ESTATE), checked["status"]
    assert np.array_equal(checked["status"], plain["status"]), (checked["status"], plain["status"])
    assert checked["rc"] == plain["rc"]
    for key in ("ttft", "ttlt", "tbtmax", "counters", "pct", "switches", "status"):
        assert np.array_equal(checked[key], plain[key]), key
    assert np.array_equal(checked["gamma"].view(np.int64), plain["gamma"].view(np.int64))
    if "assign" in plain:
        assert np.array_equal(checked["assign"], plain["assign"])


FULL_SIZE = ["1", "2", "3", "4", "4-comparators", "4-ada", "4-ladder", "4-cache", "5"]


@pytest.mark.parametrize("key", FULL_SIZE)
def test_checking_build_at_full_size(torch, key):
    """Every full-size workload with stored oracle digests, under the checking
    build: no violation in any instance, and the checked instances' digests
    equal the oracle's (the large sweep: its 508-instance subset; instances
    that fail with a latency overflow are compared by their status)."""
    import json
    import sys

    from paper_2606_18431_amd import tas

    here = os.path.dirname(os.path.abspath(__file__))
    sys.path.insert(0, os.path.join(here, "golden"))
    from digests import input_digest, instance_digests
    from make_fullsize_digests import make

    gold = json.load(open(os.path.join(here, "golden", "fullsize_digests.json")))["workloads"]
    if key not in gold:
        pytest.skip(f"no stored digests for {key}")
    ref = gold[key]
    w = make(key)
    assert input_digest(w) == ref["inputs"], "the input generator drifted"
    sel = np.asarray(ref["instances"], np.int64) if "instances" in ref else np.arange(w.n_inst)
    print(f"[gpu] checked full size {ref['name']}: {w.n_inst} x {w.n_req}", flush=True)
    prev = tas.select_library(tas.CHECK_LIB_PATH)
    try:
        sim = tas.Simulation(w)
        sim.step()
        g = sim.results(latencies=False)
        dev = sim.pct.device
        lat = [torch.empty((w.n_inst, w.n_req), dtype=torch.int32, device=dev) for _ in range(3)]
        tas.tas_latencies(sim.ctx, *lat)
        ix = torch.as_tensor(sel, device=dev)
        got = {k: t.index_select(0, ix).cpu().numpy().view(np.uint32)
               for k, t in zip(("ttft", "ttlt", "tbtmax"), lat)}
        del lat
        sim.close()
    finally:
        tas.select_library(prev)
    torch.cuda.empty_cache()
    assert not np.any(g["status"] == tas.TAS_ESTATE), np.nonzero(g["status"] == tas.TAS_ESTATE)
    assert g["rc"] == ref.get("rc", 0), tas.tas_strerror(g["rc"])
    dig = instance_digests(got["ttft"], got["ttlt"], got["tbtmax"], g["counters"][sel],
                           g["pct"][sel], g["status"][sel])
    want = ref["digests"]
    assert len(want) // 16 == len(sel)
    bad = [j for j in range(len(sel)) if dig[j] != want[16 * j:16 * (j + 1)]]
    assert not bad, f"{len(bad)} instances differ from the oracle, first {int(sel[bad[0]])}"
