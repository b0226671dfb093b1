"""Parity at the full sizes of the five workloads, in the launch configuration
the benchmark times (every instance of the sweep in one tas_run, default list
capacity), checked against the CPU oracle on a sample of instances.

The GPU simulates the whole sweep; the oracle recomputes the sampled
instances one by one. Every sampled instance must match exactly: per-request
TTFT, TTLT and maximum gap, the eight counters and the nine percentiles. The
sample covers every policy variant (FCFS, SRPT, UniBoost and vanilla boost at
the smallest and largest gamma) on the first and the last trace, plus seeded
random instances. Every instance's status must be TAS_OK.
"""
import os

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


def sample_instances(w, n_random=4, seed=0):
    if w.n_inst <= 64:  # the tiny workload: every instance
        return np.arange(w.n_inst, dtype=np.int64)
    S = w.meta["n_settings"]
    T = w.n_traces
    pick = set()
    for t in (0, T - 1):
        for s in sorted({0, 1, 2, 3, S - 2, S - 1}):
            if s < S:
                pick.add(t * S + s)
    rng = np.random.default_rng([1234, seed, w.meta["cfg"]])
    pick.update(int(i) for i in rng.choice(w.n_inst, size=min(n_random, w.n_inst), replace=False))
    return np.array(sorted(pick), np.int64)


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4, 5])
def test_full_size_sampled_parity(torch, cfg):
    from paper_2606_18431_amd import tas

    w = W.make(cfg)
    print(f"[gpu] full-size {W.NAMES[cfg]}: {w.n_inst} instances x {w.n_req} requests", flush=True)
    sim = tas.Simulation(w)
    sim.step()
    n, m = w.n_inst, w.n_req
    dev = sim.pct.device
    lat = [torch.empty((n, m), dtype=torch.int32, device=dev) for _ in range(3)]
    tas.tas_latencies(sim.ctx, *lat)
    g = sim.results(latencies=False)
    assert g["rc"] == 0, tas.tas_strerror(g["rc"])
    assert (g["status"] == 0).all()
    sel = sample_instances(w)
    idx = torch.as_tensor(sel, device=dev)
    got = {k: t.index_select(0, idx).cpu().numpy().view(np.uint32)
           for k, t in zip(("ttft", "ttlt", "tbtmax"), lat)}
    sim.close()
    del lat
    o = oracle.run(w.subset(sel), n_threads=min(16, os.cpu_count() or 1))
    assert o["rc"] == 0
    for j, i in enumerate(sel):
        for key in ("ttft", "ttlt", "tbtmax"):
            if not np.array_equal(got[key][j], o[key][j]):
                bad = np.nonzero(got[key][j] != o[key][j])[0]
                raise AssertionError(f"instance {i} {key}: {len(bad)} differ, first request "
                                     f"{bad[0]}: gpu {got[key][j][bad[0]]} oracle "
                                     f"{o[key][j][bad[0]]}")
        assert np.array_equal(g["counters"][i], o["counters"][j]), (i, g["counters"][i],
                                                                    o["counters"][j])
        assert np.array_equal(g["pct"][i], o["pct"][j]), (i, g["pct"][i], o["pct"][j])


@pytest.mark.parametrize("grid", ["ada", "ladder", "cache"])
def test_full_size_large_sweep_other_grids(torch, grid):
    """The large-sweep traces (256 x 50,000 requests) under the adaptive-gamma,
    design-phase and cache-aware settings grids (the last with seeded
    prefix-cache hits), in the launch `bench.py --grid` times (the
    extended kernel build, its default list size): every instance TAS_OK, and
    all eight settings of the first and the last trace exactly equal to the
    oracle, final adaptive gamma bit for bit."""
    from paper_2606_18431_amd import tas

    w = W.make(4, grid=grid)
    print(f"[gpu] full-size large sweep, {grid} grid: {w.n_inst} instances", flush=True)
    sim = tas.Simulation(w)
    sim.step()
    n, m = w.n_inst, w.n_req
    dev = sim.pct.device
    lat = [torch.empty((n, m), dtype=torch.int32, device=dev) for _ in range(3)]
    tas.tas_latencies(sim.ctx, *lat)
    g = sim.results(latencies=False)
    assert g["rc"] == 0, tas.tas_strerror(g["rc"])
    assert (g["status"] == 0).all()
    sel = np.concatenate([np.arange(8), np.arange(n - 8, n)])
    idx = torch.as_tensor(sel, device=dev)
    got = {k: t.index_select(0, idx).cpu().numpy().view(np.uint32)
           for k, t in zip(("ttft", "ttlt", "tbtmax"), lat)}
    sim.close()
    del lat
    o = oracle.run(w.subset(sel), n_threads=min(16, os.cpu_count() or 1))
    assert o["rc"] == 0
    for j, i in enumerate(sel):
        for key in ("ttft", "ttlt", "tbtmax"):
            assert np.array_equal(got[key][j], o[key][j]), (i, key)
        assert np.array_equal(g["counters"][i], o["counters"][j]), i
        assert np.array_equal(g["pct"][i], o["pct"][j]), i
        assert g["switches"][i] == o["switches"][j], i
        assert g["gamma"][i:i + 1].view(np.int64)[0] == o["gamma"][j:j + 1].view(np.int64)[0], i


def replay_router_fast(arrival, assign, ttlt, R):
    """Every request went to a replica holding the fewest requests not
    completed by its arrival (ties to the lowest), checked for all N at once:
    at a_j replica r holds the requests dispatched to it before j minus those
    of them completed by a_j (a completion is never before its arrival, so
    none of the later ones has completed by then)."""
    a = np.asarray(arrival, np.int64)
    done = a + np.asarray(ttlt, np.int64)
    n = len(a)
    held = np.zeros((R, n), np.int64)
    for r in range(R):
        mine = assign == r
        before = np.concatenate([[0], np.cumsum(mine)[:-1]])
        fin = np.sort(done[mine])
        held[r] = before - np.searchsorted(fin, a, side="right")
    return bool(np.all(np.argmin(held, axis=0) == assign))


def test_full_size_jsq_clusters(torch):
    """The JSQ bench configuration (large-sweep law, 32 clusters x 8 replicas,
    50,000 requests per cluster, FCFS / UniBoost / vanilla boost / Sarathi) in
    its launch: every instance TAS_OK; on the first and the last cluster,
    every routing decision agrees with the GPU's own completion times, and
    every replica's requests, simulated by the oracle as a plain instance,
    give exactly the GPU's latencies and the replica's counters."""
    from paper_2606_18431_amd import tas

    R = 8
    w = W.make_cluster(4, n_clusters=32, replicas=R, dispatch="jsq", n_req=50000 // R)
    print(f"[gpu] full-size jsq: {w.n_inst} clusters x {R} replicas x {w.n_req} requests",
          flush=True)
    sim = tas.Simulation(w)
    sim.step()
    g = sim.results()
    sim.close()
    assert g["rc"] == 0, tas.tas_strerror(g["rc"])
    assert (g["status"] == 0).all()
    S = w.meta["n_settings"]
    sel = list(range(S)) + list(range(w.n_inst - S, w.n_inst))
    jobs = []
    for i in sel:
        t = int(w.settings["trace"][i])
        assert replay_router_fast(w.arrival_us[t], g["assign"][i], g["ttlt"][i], R), i
        for r in range(R):
            idx = np.nonzero(g["assign"][i] == r)[0]
            jobs.append((i, r, idx))
    def check(job):
        i, r, idx = job
        t = int(w.settings["trace"][i])
        st = w.settings[i:i + 1].copy()
        st["trace"] = 0  # the replica's requests are the one trace of `one`
        one = W.Workload("replica", w.arrival_us[t][idx][None], w.prompt[t][idx][None],
                         w.decode[t][idx][None], w.engine, st)
        o = oracle.run(one, n_threads=1)
        assert o["rc"] == 0, (i, r)
        for key in ("ttft", "ttlt", "tbtmax"):
            assert np.array_equal(o[key][0], g[key][i][idx]), (i, r, key)
        assert np.array_equal(o["counters"][0], g["rcounters"][i, r]), (i, r)

    from concurrent.futures import ThreadPoolExecutor

    with ThreadPoolExecutor(min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(check, jobs))
